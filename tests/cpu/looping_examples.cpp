// The kernel-looping pass (paper_2410_23668_amd/looping) on the worked
// examples of Sec. 3.3 (Fig. 8 (a)-(d)), on a toy decoder, on cases that
// must not be chained or must not match, and on seeded random programs.
// For every program: the pass's analysis and rewrite are printed as one JSON
// object per line (compared with the paper's values by the Python test), and
// the original and the rewritten program are both run by the interpreter on
// seeded inputs: every tensor live at the end must come out bit-identical
// ("equivalent"), and a chained intermediate that the rewrite keeps on chip
// must never be written ("untouched").
// Usage: looping_examples [--fuzz N]
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <string>
#include <vector>

#include "kl_looping.h"

using namespace klp;

namespace {

uint64_t mix(uint64_t x) {   // SplitMix64 output function
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

Memory seeded(const Program &p, uint64_t seed) {
    Memory m;
    for (size_t t = 0; t < p.tensors.size(); ++t) {
        std::vector<double> v((size_t)p.tensors[t].rows * p.tensors[t].cols);
        for (size_t i = 0; i < v.size(); ++i)   // small integers and halves: exact sums
            v[i] = (double)((int)(mix(seed ^ (t << 32) ^ i) % 9) - 4) * 0.5;
        m.push_back(v);
    }
    return m;
}

int tensor(Program &p, const std::string &name, int rows, int cols) {
    p.tensors.push_back({name, rows, cols});
    return (int)p.tensors.size() - 1;
}

int find(const Program &p, const std::string &name) {
    for (size_t i = 0; i < p.tensors.size(); ++i)
        if (p.tensors[i].name == name) return (int)i;
    std::fprintf(stderr, "no tensor %s\n", name.c_str());
    std::exit(2);
}

void call(Program &p, int kernel, const std::vector<std::string> &args) {
    Call c;
    c.kernel = kernel;
    for (const std::string &a : args) c.args.push_back({find(p, a)});
    p.calls.push_back(c);
}

std::string names(const Program &p, const std::vector<int> &ts) {
    std::string s = "[";
    for (size_t i = 0; i < ts.size(); ++i)
        s += (i ? ", " : "") + std::string("\"") + p.tensors[ts[i]].name + "\"";
    return s + "]";
}

std::string esc(const std::string &s) {
    std::string o;
    for (char c : s) {
        if (c == '"' || c == '\\') o += '\\';
        if (c == '\n') { o += "\\n"; continue; }
        o += c;
    }
    return o;
}

// kernels of Fig. 8
Kernel kernel_a(int n) {   // z += x * y, elementwise
    Kernel k;
    k.name = "kernel_a";
    k.params = {{"x", n, 1}, {"y", n, 1}, {"z", n, 1}};
    k.body = {accumulate(param(2), emul(leaf(param(0)), leaf(param(1))))};
    return k;
}
Kernel kernel_b(int n) {   // z = y - x
    Kernel k;
    k.name = "kernel_b";
    k.params = {{"x", n, 1}, {"y", n, 1}, {"z", n, 1}};
    k.body = {assign(param(2), sub(leaf(param(1)), leaf(param(0))))};
    return k;
}
Kernel kernel_c(int m, int n) {   // z = w x
    Kernel k;
    k.name = "kernel_c";
    k.params = {{"w", m, m}, {"x", m, n}, {"z", m, n}};
    k.body = {assign(param(2), matmul(leaf(param(0)), leaf(param(1))))};
    return k;
}
Kernel kernel_d(int m, int n, int t, int rows_written) {   // z[t:t+T] = w[t:t+T] x, tiled
    Kernel k;
    k.name = rows_written == m ? "kernel_d" : "kernel_half";
    k.params = {{"w", m, m}, {"x", m, n}, {"z", m, n}};
    k.body = {loop(0, 0, rows_written, t,
                   {assign(rows(param(2), 0, 0, 1, t),
                           matmul(leaf(rows(param(0), 0, 0, 1, t)), leaf(param(1))))})};
    return k;
}
// a decoder layer: h = (wa x) .* cs; kv += h; y = wb h + x
Kernel layer(int h) {
    Kernel k;
    k.name = "layer";
    k.params = {{"wa", h, h}, {"wb", h, h}, {"cs", h, 1}, {"x", h, 1}, {"y", h, 1}, {"kv", h, 1}};
    k.locals = {{"h", h, 1}};
    k.body = {assign(local(0), emul(matmul(leaf(param(0)), leaf(param(3))), leaf(param(2)))),
              accumulate(param(5), leaf(local(0))),
              assign(param(4), add(matmul(leaf(param(1)), leaf(local(0))), leaf(param(3))))};
    return k;
}

struct Result {
    bool equivalent = true, untouched = true;
    int calls_after = 0;
};

// Runs the pass on p, prints its JSON line, checks the rewritten program.
Result report(const char *name, const Program &p, uint64_t seed, bool print) {
    PassReport rep;
    const Program q = kernel_looping_pass(p, &rep);
    const Memory init = seeded(p, seed);
    const Memory a = run_program(p, init), b = run_program(q, init);
    Result r;
    r.calls_after = (int)q.calls.size();
    for (int t : p.outputs)
        if (std::memcmp(a[t].data(), b[t].data(), a[t].size() * sizeof(double)) != 0)
            r.equivalent = false;
    // a chained intermediate not live after its chain stays on chip: the
    // collapsed call never writes it (other calls may)
    int removed = 0;
    for (size_t c = 0; c < rep.collapsed.size(); ++c) {
        const Candidate &cd = rep.collapsed[c];
        const int qi = cd.first - removed;   // the collapsed call's index in q
        removed += cd.count - 1;
        Program before = q, through = q;
        before.calls.resize(qi);
        through.calls.resize(qi + 1);
        const Memory m0 = run_program(before, init), m1 = run_program(through, init);
        for (const Rewrite::Buffer &bf : rep.rewrites[c].buffers) {
            if (cd.P[bf.out_param] != (kLocal | kOut)) continue;
            for (int n = 0; n + 1 < cd.count; ++n) {
                const int t = p.calls[cd.first + n].args[bf.out_param][0];
                if (std::memcmp(m0[t].data(), m1[t].data(), m1[t].size() * sizeof(double)) != 0)
                    r.untouched = false;
            }
        }
    }
    if (!print) return r;
    const std::vector<std::set<int>> LA = live_after(p);
    std::string s = std::string("{\"example\": \"") + name + "\", \"calls_before\": " +
                    std::to_string(p.calls.size()) + ", \"calls_after\": " +
                    std::to_string(q.calls.size()) + ", \"equivalent\": " +
                    (r.equivalent ? "true" : "false") + ", \"untouched\": " +
                    (r.untouched ? "true" : "false") + ", \"loops\": [";
    removed = 0;   // calls the earlier collapses removed
    for (size_t c = 0; c < rep.collapsed.size(); ++c) {
        const Candidate &cd = rep.collapsed[c];
        const Rewrite &rw = rep.rewrites[c];
        const Kernel &k = p.kernels[p.calls[cd.first].kernel];
        const int qi = cd.first - removed;
        removed += cd.count - 1;
        const int last = cd.first + cd.count - 1;
        std::vector<int> la(LA[last].begin(), LA[last].end());
        s += std::string(c ? ", " : "") + "{\"kernel\": \"" + k.name + "\", \"first\": " +
             std::to_string(cd.first) + ", \"count\": " + std::to_string(cd.count) +
             ", \"live_after\": " + names(p, la) + ", \"props\": {";
        for (size_t i = 0; i < k.params.size(); ++i)
            s += std::string(i ? ", " : "") + "\"" + k.params[i].name + "\": \"" +
                 prop_string(cd.P[i]) + "\"";
        s += "}, \"grouped\": [";
        bool first = true;
        for (size_t i = 0; i < k.params.size(); ++i)
            if (cd.grouped[i]) {
                s += std::string(first ? "" : ", ") + "\"" + k.params[i].name + "\"";
                first = false;
            }
        s += "], \"call\": [";
        for (size_t i = 0; i < rw.call.args.size(); ++i)
            s += std::string(i ? ", " : "") + names(p, rw.call.args[i]);
        s += "], \"buffers\": [";
        for (size_t i = 0; i < rw.buffers.size(); ++i)
            s += std::string(i ? ", " : "") + "{\"in\": \"" +
                 k.params[rw.buffers[i].in_param].name + "\", \"out\": \"" +
                 k.params[rw.buffers[i].out_param].name + "\", \"double\": " +
                 (rw.buffers[i].double_buffered ? "true" : "false") + "}";
        s += "], \"stores_each_iteration\": [";
        for (size_t i = 0; i < rw.stores_each_iteration.size(); ++i)
            s += std::string(i ? ", " : "") + "\"" + k.params[rw.stores_each_iteration[i]].name +
                 "\"";
        s += "], \"stores_at_end\": [";
        for (size_t i = 0; i < rw.stores_at_end.size(); ++i)
            s += std::string(i ? ", " : "") + "\"" + k.params[rw.stores_at_end[i]].name + "\"";
        s += "], \"printed\": \"" + esc(print_kernel(rw.kernel)) + "\", \"printed_call\": \"" +
             esc(print_call(q, q.calls[qi])) + "\"}";
    }
    s += "]}";
    std::printf("%s\n", s.c_str());
    return r;
}

// ------------------------------------------------------------- the programs
Program example_a() {
    Program p;
    p.kernels = {kernel_a(5)};
    for (const char *t : {"a", "b", "c", "d", "e", "f"}) tensor(p, t, 5, 1);
    call(p, 0, {"a", "b", "c"});
    call(p, 0, {"a", "e", "f"});
    p.outputs = {find(p, "c"), find(p, "f")};
    return p;
}
Program example_b() {
    Program p;
    p.kernels = {kernel_b(5)};
    for (const char *t : {"a", "b", "c", "d", "e", "f", "g"}) tensor(p, t, 5, 1);
    call(p, 0, {"a", "b", "c"});
    call(p, 0, {"c", "d", "e"});
    call(p, 0, {"f", "e", "g"});
    p.outputs = {find(p, "c"), find(p, "e"), find(p, "g")};
    return p;
}
Program example_c() {
    Program p;
    p.kernels = {kernel_c(4, 3)};
    tensor(p, "w0", 4, 4);
    tensor(p, "w1", 4, 4);
    for (const char *t : {"x", "y", "z"}) tensor(p, t, 4, 3);
    call(p, 0, {"w0", "x", "y"});
    call(p, 0, {"w1", "y", "z"});
    p.outputs = {find(p, "z")};
    return p;
}
Program example_d() {
    Program p;
    p.kernels = {kernel_d(4, 3, 2, 4)};
    for (const char *t : {"w0", "w1", "w2"}) tensor(p, t, 4, 4);
    for (const char *t : {"x", "y", "z", "r"}) tensor(p, t, 4, 3);
    call(p, 0, {"w0", "x", "y"});
    call(p, 0, {"w1", "y", "z"});
    call(p, 0, {"w2", "z", "r"});
    p.outputs = {find(p, "y"), find(p, "z"), find(p, "r")};
    return p;
}
// L layers; dump_hidden: every layer's output is live after the chain
Program decoder(int L, bool dump_hidden) {
    Program p;
    const int H = 6;
    p.kernels = {layer(H)};
    for (int l = 0; l < L; ++l) {
        tensor(p, "wa" + std::to_string(l), H, H);
        tensor(p, "wb" + std::to_string(l), H, H);
        tensor(p, "kv" + std::to_string(l), H, 1);
    }
    tensor(p, "cs", H, 1);
    for (int l = 0; l <= L; ++l) tensor(p, "x" + std::to_string(l), H, 1);
    for (int l = 0; l < L; ++l)
        call(p, 0, {"wa" + std::to_string(l), "wb" + std::to_string(l), "cs",
                    "x" + std::to_string(l), "x" + std::to_string(l + 1), "kv" + std::to_string(l)});
    p.outputs.insert(find(p, "x" + std::to_string(L)));
    for (int l = 0; l < L; ++l) {
        p.outputs.insert(find(p, "kv" + std::to_string(l)));
        if (dump_hidden && l > 0) p.outputs.insert(find(p, "x" + std::to_string(l)));
    }
    return p;
}
// the same output tensor in every call: {Const} with {Out} is the top
Program same_output() {
    Program p;
    p.kernels = {kernel_a(5)};
    for (const char *t : {"a", "b", "c", "d", "e"}) tensor(p, t, 5, 1);
    call(p, 0, {"a", "b", "c"});
    call(p, 0, {"d", "e", "c"});
    p.outputs = {find(p, "c")};
    return p;
}
// a chain whose writes cover half of what the next call reads: not Local
Program half_write() {
    Program p;
    p.kernels = {kernel_d(4, 3, 2, 2)};
    for (const char *t : {"w0", "w1"}) tensor(p, t, 4, 4);
    for (const char *t : {"x", "y", "z"}) tensor(p, t, 4, 3);
    call(p, 0, {"w0", "x", "y"});
    call(p, 0, {"w1", "y", "z"});
    p.outputs = {find(p, "z")};
    return p;
}
// a chain x -> y -> x -> y: the intermediate y is named again two calls
// later, so the pair is not uniquely chained
Program ping_pong() {
    Program p;
    p.kernels = {kernel_c(4, 3)};
    for (const char *t : {"w0", "w1", "w2"}) tensor(p, t, 4, 4);
    for (const char *t : {"x", "y"}) tensor(p, t, 4, 3);
    call(p, 0, {"w0", "x", "y"});
    call(p, 0, {"w1", "y", "x"});
    call(p, 0, {"w2", "x", "y"});
    p.outputs = {find(p, "y")};
    return p;
}
// the greedy driver over runs of three kernels
Program mixed() {
    Program p;
    p.kernels = {kernel_c(4, 3), kernel_a(5), kernel_b(5)};
    for (const char *t : {"w0", "w1", "w2"}) tensor(p, t, 4, 4);
    for (const char *t : {"x0", "x1", "x2", "x3"}) tensor(p, t, 4, 3);
    for (const char *t : {"a", "b", "c", "d", "e", "f", "g"}) tensor(p, t, 5, 1);
    call(p, 0, {"w0", "x0", "x1"});
    call(p, 0, {"w1", "x1", "x2"});
    call(p, 0, {"w2", "x2", "x3"});
    call(p, 1, {"a", "b", "c"});
    call(p, 2, {"c", "d", "e"});
    call(p, 2, {"e", "f", "g"});
    p.outputs = {find(p, "x3"), find(p, "g")};
    return p;
}

// Random programs: runs of calls to four kernels over a small tensor pool,
// often chained, with random outputs.
Program random_program(uint64_t seed) {
    Program p;
    p.kernels = {kernel_a(5), kernel_b(5), kernel_c(4, 3), kernel_d(4, 3, 2, 4)};
    uint64_t s = seed;
    auto rnd = [&](int n) { s = mix(s); return (int)(s % (uint64_t)n); };
    std::vector<int> vec, mat, sq;
    for (int i = 0; i < 7; ++i) vec.push_back(tensor(p, "v" + std::to_string(i), 5, 1));
    for (int i = 0; i < 7; ++i) mat.push_back(tensor(p, "m" + std::to_string(i), 4, 3));
    for (int i = 0; i < 4; ++i) sq.push_back(tensor(p, "w" + std::to_string(i), 4, 4));
    const int ncalls = 6 + rnd(10);
    int prev_kernel = -1, prev_out = -1;
    for (int c = 0; c < ncalls; ++c) {
        const int k = (prev_kernel >= 0 && rnd(3) != 0) ? prev_kernel : rnd(4);
        const std::vector<int> &pool = k < 2 ? vec : mat;
        Call call;
        call.kernel = k;
        std::vector<int> used;
        auto pick = [&](const std::vector<int> &pl) {
            int t;
            do t = pl[rnd((int)pl.size())];
            while (std::find(used.begin(), used.end(), t) != used.end());
            used.push_back(t);
            return t;
        };
        // chain: the previous call's output as this call's input (x, or y
        // for the elementwise kernels now and then)
        const bool chain = k == prev_kernel && rnd(4) != 0;
        const int in_slot = (k < 2 && rnd(3) == 0) ? 1 : (k < 2 ? 0 : 1);
        std::vector<int> args(3, -1);
        if (chain) {
            args[in_slot] = prev_out;
            used.push_back(prev_out);
        }
        for (int i = 0; i < 3; ++i)
            if (args[i] < 0) args[i] = (k >= 2 && i == 0) ? pick(sq) : pick(pool);
        for (int a : args) call.args.push_back({a});
        p.calls.push_back(call);
        prev_kernel = k;
        prev_out = args[2];
    }
    for (size_t t = 0; t < p.tensors.size(); ++t)
        if (rnd(2)) p.outputs.insert((int)t);
    return p;
}

// ------------------------------------------------- planted mistakes (test side)
// Each builds the rewrite a pass with one of its conditions left out would
// make, and reports whether running it changes a live output (it must).

void retarget(std::vector<Stmt> &body, int from, int to) {
    for (Stmt &s : body) {
        if (s.kind == Stmt::kLoop) {
            retarget(s.body, from, to);
            continue;
        }
        if (s.dst.base == Ref::kBuffer && s.dst.id == from) s.dst.id = to;
        std::function<ExprP(const ExprP &)> m = [&](const ExprP &e) -> ExprP {
            if (e->op == Expr::kLeaf) {
                Ref r = e->ref;
                if (r.base == Ref::kBuffer && r.id == from) r.id = to;
                return leaf(r);
            }
            auto n = std::make_shared<Expr>(*e);
            n->a = m(e->a);
            n->b = m(e->b);
            return n;
        };
        s.rhs = m(s.rhs);
    }
}

bool outputs_differ(const Program &p, const Program &q, uint64_t seed) {
    const Memory init = seeded(p, seed);
    const Memory a = run_program(p, init), b = run_program(q, init);
    for (int t : p.outputs)
        if (std::memcmp(a[t].data(), b[t].data(), a[t].size() * sizeof(double)) != 0) return true;
    return false;
}

Program with_rewrite(const Program &p, const Candidate &c, Rewrite rw) {
    Program q;
    q.tensors = p.tensors;
    q.kernels = p.kernels;
    q.outputs = p.outputs;
    for (int i = 0; i < c.first; ++i) q.calls.push_back(p.calls[i]);
    rw.call.kernel = (int)q.kernels.size();
    q.kernels.push_back(rw.kernel);
    q.calls.push_back(rw.call);
    for (size_t i = c.first + c.count; i < p.calls.size(); ++i) q.calls.push_back(p.calls[i]);
    return q;
}

// example (d) with one buffer where the pass double-buffers: the tiles of a
// product overwrite rows of its input that later tiles still read
bool planted_single_buffer() {
    const Program p = example_d();
    const Candidate c = analyse(p, 0, 3, live_after(p)[2]);
    Rewrite rw = rewrite(p, c);
    if (rw.buffers.size() != 1 || !rw.buffers[0].double_buffered) return false;
    // drop "buf0 = buf1" (the first statement after the tile loop) and let
    // the tiles write buf0
    std::vector<Stmt> &iter = rw.kernel.body[1].body;
    iter.erase(iter.begin() + 1);
    retarget(rw.kernel.body, 1, 0);
    return outputs_differ(p, with_rewrite(p, c, rw), 11);
}

// a chain whose intermediate another call of the list reads: c = b - a,
// e = d - c, g = c - e; kept on chip, the last call reads a stale c
Program reread_chain() {
    Program p;
    p.kernels = {kernel_b(5)};
    for (const char *t : {"a", "b", "c", "d", "e", "g"}) tensor(p, t, 5, 1);
    call(p, 0, {"a", "b", "c"});
    call(p, 0, {"c", "d", "e"});
    call(p, 0, {"e", "c", "g"});
    p.outputs = {find(p, "g")};
    return p;
}
bool planted_chain_without_uniqueness() {
    const Program p = reread_chain();
    Candidate c = analyse(p, 0, 3, live_after(p)[2]);
    if (c.P[0] & kLocal) return false;   // the pass itself must not chain it
    c.P[0] = kIn | kLocal;
    c.P[2] = kLocal | kOut;
    c.partner[0] = 2;
    c.partner[2] = 0;
    c.grouped[0] = c.grouped[2] = false;
    return outputs_differ(p, with_rewrite(p, c, rewrite(p, c)), 12);
}

}  // namespace

int main(int argc, char **argv) {
    int fuzz = 0;
    for (int i = 1; i < argc; ++i)
        if (!std::strcmp(argv[i], "--fuzz") && i + 1 < argc) fuzz = std::atoi(argv[++i]);
    report("a", example_a(), 1, true);
    report("b", example_b(), 2, true);
    report("c", example_c(), 3, true);
    report("d", example_d(), 4, true);
    report("decoder", decoder(4, false), 5, true);
    report("decoder_dump_hidden", decoder(4, true), 6, true);
    report("same_output", same_output(), 7, true);
    report("half_write", half_write(), 8, true);
    report("ping_pong", ping_pong(), 9, true);
    report("mixed", mixed(), 10, true);
    report("reread_chain", reread_chain(), 13, true);
    std::printf("{\"planted_single_buffer_detected\": %s, "
                "\"planted_chain_without_uniqueness_detected\": %s}\n",
                planted_single_buffer() ? "true" : "false",
                planted_chain_without_uniqueness() ? "true" : "false");
    // lattice: every join against an independent reading (the smallest
    // element containing the union of the two sets, or the top)
    int lattice_bad = 0;
    std::vector<PropSet> el = lattice_elements();
    for (PropSet a : el)
        for (PropSet b : el) {
            PropSet want = kTop;
            for (PropSet u : el)
                if ((u & (a | b)) == (a | b) && (want == kTop || __builtin_popcount(u) <
                                                                     __builtin_popcount(want)))
                    want = u;
            if (lattice_join(a, b) != want || lattice_join(b, a) != want) ++lattice_bad;
            for (PropSet c : el)
                if (lattice_join(lattice_join(a, b), c) != lattice_join(a, lattice_join(b, c)))
                    ++lattice_bad;
        }
    std::printf("{\"lattice_mismatches\": %d}\n", lattice_bad);
    if (fuzz) {
        int bad = 0, loops = 0, buffers = 0, dbl = 0, live_stores = 0, end_stores = 0;
        for (int i = 0; i < fuzz; ++i) {
            const Program p = random_program(1000 + i);
            PassReport rep;
            kernel_looping_pass(p, &rep);
            const Result r = report("fuzz", p, 77 + i, false);
            if (!r.equivalent || !r.untouched) {
                ++bad;
                if (bad <= 3) report("fuzz_failure", p, 77 + i, true);
            }
            loops += (int)rep.rewrites.size();
            for (const Rewrite &rw : rep.rewrites) {
                buffers += (int)rw.buffers.size();
                for (const auto &b : rw.buffers) dbl += b.double_buffered;
                live_stores += (int)rw.stores_each_iteration.size();
                end_stores += (int)rw.stores_at_end.size();
            }
        }
        std::printf("{\"fuzz_programs\": %d, \"fuzz_failures\": %d, \"looped_kernels\": %d, "
                    "\"buffers\": %d, \"double_buffers\": %d, \"stores_each_iteration\": %d, "
                    "\"stores_at_end\": %d}\n",
                    fuzz, bad, loops, buffers, dbl, live_stores, end_stores);
    }
    return 0;
}
