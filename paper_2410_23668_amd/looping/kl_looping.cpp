// Kernel looping as a compiler pass over a small kernel-call IR (Sec. 3).
// See kl_looping.h for the IR and the steps.
#include "kl_looping.h"

#include <algorithm>
#include <functional>
#include <sstream>
#include <stdexcept>

namespace klp {

// ===================================================================== lattice
//
// Fig. 6b: the empty set at the bottom, the five singletons above it, the
// elements (1)-(7) above those, the top above (1), (2), (6) and (7).  Each
// element is written as the set of usage properties it stands for, which the
// figure's edges fix: (1) covers {Const} and {In}, (2) {In} and {Local}, (3)
// {In} and {Live}, (4) {Local} and {Out}, (5) {Live} and {Out}, (6) covers (3)
// and (5), (7) covers (4) and (5).
namespace {

constexpr PropSet kE1 = kConst | kIn, kE2 = kIn | kLocal, kE3 = kIn | kLive,
                  kE4 = kLocal | kOut, kE5 = kLive | kOut, kE6 = kIn | kLive | kOut,
                  kE7 = kLocal | kLive | kOut;

struct Edge { PropSet lo, hi; };
const std::vector<Edge> &hasse() {
    static const std::vector<Edge> e = {
        {0, kConst}, {0, kIn}, {0, kLocal}, {0, kLive}, {0, kOut},
        {kConst, kE1}, {kIn, kE1}, {kIn, kE2}, {kIn, kE3},
        {kOut, kE4}, {kOut, kE5}, {kLocal, kE2}, {kLocal, kE4},
        {kLive, kE3}, {kLive, kE5},
        {kE3, kE6}, {kE5, kE6}, {kE4, kE7}, {kE5, kE7},
        {kE1, kTop}, {kE2, kTop}, {kE6, kTop}, {kE7, kTop},
    };
    return e;
}

// a <= b: b is reachable from a going up the diagram
bool leq(PropSet a, PropSet b) {
    if (a == b) return true;
    for (const Edge &e : hasse())
        if (e.lo == a && leq(e.hi, b)) return true;
    return false;
}

}  // namespace

const std::vector<PropSet> &lattice_elements() {
    static const std::vector<PropSet> v = {0,   kConst, kIn, kLocal, kLive, kOut, kE1,
                                           kE2, kE3,    kE4, kE5,    kE6,   kE7};
    return v;
}

PropSet lattice_join(PropSet a, PropSet b) {
    std::vector<PropSet> all = lattice_elements();
    all.push_back(kTop);
    std::vector<PropSet> ub;
    for (PropSet u : all)
        if (leq(a, u) && leq(b, u)) ub.push_back(u);
    for (PropSet u : ub) {
        bool least = true;
        for (PropSet v : ub) least = least && leq(u, v);
        if (least) return u;
    }
    throw std::logic_error("lattice_join: no least upper bound");
}

std::string prop_string(PropSet p) {
    if (p == kTop) return "T";
    static const char *names[] = {"Const", "In", "Local", "Live", "Out"};
    std::string s = "{";
    for (int i = 0; i < 5; ++i)
        if (p & (1u << i)) s += (s.size() > 1 ? "," : "") + std::string(names[i]);
    return s + "}";
}

// ===================================================================== builders
Ref param(int id) {
    Ref r;
    r.base = Ref::kParam;
    r.id = id;
    return r;
}
Ref local(int id) {
    Ref r;
    r.base = Ref::kLocalTensor;
    r.id = id;
    return r;
}
Ref rows(Ref r, int lo_const, int lo_var, int lo_step, int len) {
    r.sliced = true;
    r.lo_const = lo_const;
    r.lo_var = lo_var;
    r.lo_step = lo_step;
    r.len = len;
    return r;
}
static ExprP node(Expr::Op op, ExprP a, ExprP b) {
    auto e = std::make_shared<Expr>();
    e->op = op;
    e->a = std::move(a);
    e->b = std::move(b);
    return e;
}
ExprP leaf(const Ref &r) {
    auto e = std::make_shared<Expr>();
    e->op = Expr::kLeaf;
    e->ref = r;
    return e;
}
ExprP add(ExprP a, ExprP b) { return node(Expr::kAdd, std::move(a), std::move(b)); }
ExprP sub(ExprP a, ExprP b) { return node(Expr::kSub, std::move(a), std::move(b)); }
ExprP emul(ExprP a, ExprP b) { return node(Expr::kEMul, std::move(a), std::move(b)); }
ExprP matmul(ExprP a, ExprP b) { return node(Expr::kMatMul, std::move(a), std::move(b)); }
Stmt assign(const Ref &dst, ExprP rhs) {
    Stmt s;
    s.kind = Stmt::kAssign;
    s.dst = dst;
    s.rhs = std::move(rhs);
    return s;
}
Stmt accumulate(const Ref &dst, ExprP rhs) {
    Stmt s = assign(dst, std::move(rhs));
    s.kind = Stmt::kAccumulate;
    return s;
}
Stmt loop(int var, int lo, int hi, int step, std::vector<Stmt> body) {
    Stmt s;
    s.kind = Stmt::kLoop;
    s.var = var;
    s.lo = lo;
    s.hi = hi;
    s.step = step;
    s.body = std::move(body);
    return s;
}

// ===================================================================== usage
namespace {

using Vars = std::map<int, int>;

int var_value(const Vars &v, int id) {
    const auto it = v.find(id);
    if (it == v.end()) throw std::runtime_error("loop variable used outside its loop");
    return it->second;
}

// rows [lo, hi) of a reference to a tensor with 'nrows' rows
std::pair<int, int> ref_rows(const Ref &r, int nrows, const Vars &v) {
    if (!r.sliced) return {0, nrows};
    const int lo = r.lo_const + (r.lo_var >= 0 ? r.lo_step * var_value(v, r.lo_var) : 0);
    if (lo < 0 || lo + r.len > nrows) throw std::runtime_error("row slice out of range");
    return {lo, lo + r.len};
}

// One executed access of a parameter: statement sequence number, rows.
struct Access {
    int seq;
    bool write;
    int param;
    int lo, hi;
};

void collect_expr(const Expr &e, const Kernel &k, const Vars &v, int seq,
                  std::vector<Access> &out) {
    if (e.op == Expr::kLeaf) {
        if (e.ref.base == Ref::kParam) {
            const auto rr = ref_rows(e.ref, k.params[e.ref.id].rows, v);
            out.push_back({seq, false, e.ref.id, rr.first, rr.second});
        }
        return;
    }
    collect_expr(*e.a, k, v, seq, out);
    collect_expr(*e.b, k, v, seq, out);
}

void collect(const std::vector<Stmt> &body, const Kernel &k, Vars &v, int &seq,
             std::vector<Access> &out) {
    for (const Stmt &s : body) {
        if (s.kind == Stmt::kLoop) {
            for (int i = s.lo; i < s.hi; i += s.step) {
                v[s.var] = i;
                collect(s.body, k, v, seq, out);
            }
            v.erase(s.var);
            continue;
        }
        const int my = seq++;
        collect_expr(*s.rhs, k, v, my, out);
        if (s.dst.base == Ref::kParam) {
            const auto rr = ref_rows(s.dst, k.params[s.dst.id].rows, v);
            if (s.kind == Stmt::kAccumulate)   // dst += rhs reads dst
                out.push_back({my, false, s.dst.id, rr.first, rr.second});
            out.push_back({my, true, s.dst.id, rr.first, rr.second});
        }
    }
}

std::vector<Access> accesses(const Kernel &k) {
    std::vector<Access> out;
    Vars v;
    int seq = 0;
    collect(k.body, k, v, seq, out);
    return out;
}

}  // namespace

Usage usage_of(const Kernel &k) {
    Usage u;
    u.read_rows.assign(k.params.size(), {});
    u.write_rows.assign(k.params.size(), {});
    for (const Access &a : accesses(k))
        for (int r = a.lo; r < a.hi; ++r)
            (a.write ? u.write_rows : u.read_rows)[a.param].insert(r);
    return u;
}

// ===================================================================== liveness
std::vector<std::set<int>> live_after(const Program &prog) {
    const int n = (int)prog.calls.size();
    std::vector<std::set<int>> after(n);
    std::set<int> live = prog.outputs;
    for (int c = n - 1; c >= 0; --c) {
        after[c] = live;
        const Call &call = prog.calls[c];
        const Kernel &k = prog.kernels[call.kernel];
        const Usage u = usage_of(k);
        // a call kills the tensors it overwrites whole without reading them,
        // then generates the ones it reads
        for (size_t p = 0; p < k.params.size(); ++p)
            if (u.writes((int)p) && !u.reads((int)p) &&
                (int)u.write_rows[p].size() == k.params[p].rows && call.args[p].size() == 1)
                live.erase(call.args[p][0]);
        for (size_t p = 0; p < k.params.size(); ++p)
            if (u.reads((int)p))
                for (int t : call.args[p]) live.insert(t);
    }
    return after;
}

// ===================================================================== analysis
Candidate analyse(const Program &prog, int first, int count, const std::set<int> &live_last) {
    if (count < 2) throw std::invalid_argument("analyse: a candidate has two calls or more");
    const int kid = prog.calls[first].kernel;
    const Kernel &k = prog.kernels[kid];
    const int M = (int)k.params.size(), N = count;
    std::vector<std::vector<int>> A(M, std::vector<int>(N));
    for (int c = 0; c < N; ++c) {
        const Call &call = prog.calls[first + c];
        if (call.kernel != kid) throw std::invalid_argument("analyse: calls to different kernels");
        for (int i = 0; i < M; ++i) {
            if (call.args[i].size() != 1) throw std::invalid_argument("analyse: grouped argument");
            A[i][c] = call.args[i][0];
        }
    }
    const Usage U = usage_of(k);
    Candidate C;
    C.first = first;
    C.count = count;
    C.P.assign(M, 0);
    C.partner.assign(M, -1);
    C.grouped.assign(M, false);

    // j's argument at call c is i's at call c + 1, for every c < N - 1
    auto shifted = [&](int j, int i) {
        for (int c = 0; c + 1 < N; ++c)
            if (A[j][c] != A[i][c + 1]) return false;
        return true;
    };
    // Local, read side (Fig. 6a): the unique j feeding i from the previous call
    auto read_partner = [&](int i) {
        if (!U.reads(i)) return -1;
        int found = -1, n = 0;
        for (int j = 0; j < M; ++j)
            if (j != i && shifted(j, i)) found = j, ++n;
        return n == 1 ? found : -1;
    };
    // Local, write side: the unique j reading i's argument in the next call,
    // no other parameter of the next call taking it, and i's writes covering
    // j's reads; and (the requirement that the chained tensor is used by the
    // next call only) no other call of the list naming it
    auto write_partner = [&](int i) {
        if (!U.writes(i)) return -1;
        int found = -1, n = 0;
        for (int j = 0; j < M; ++j)
            if (j != i && shifted(i, j)) found = j, ++n;
        if (n != 1) return -1;
        const int j = found;
        for (int c = 0; c + 1 < N; ++c)
            for (int h = 0; h < M; ++h)
                if (h != j && A[i][c] == A[h][c + 1]) return -1;
        for (int c = 0; c + 1 < N; ++c)
            for (int m = 0; m < N; ++m)
                if (m != c && m != c + 1)
                    for (int h = 0; h < M; ++h)
                        if (A[h][m] == A[i][c]) return -1;
        if (k.params[i].rows != k.params[j].rows || k.params[i].cols != k.params[j].cols)
            return -1;
        for (int r : U.read_rows[j])
            if (!U.write_rows[i].count(r)) return -1;
        return j;
    };
    std::vector<int> rp(M), wp(M);
    for (int i = 0; i < M; ++i) {
        rp[i] = read_partner(i);
        wp[i] = write_partner(i);
    }
    for (int i = 0; i < M; ++i) {
        std::set<int> args(A[i].begin(), A[i].end());
        const bool is_const = args.size() == 1;
        const bool is_in = U.reads(i), is_out = U.writes(i);
        // Local holds for both ends of a chained pair, or for neither
        const bool local_in = rp[i] >= 0 && wp[rp[i]] == i;
        const bool local_out = wp[i] >= 0 && rp[wp[i]] == i;
        bool is_live = false;
        if (is_out)
            for (int c = 0; c + 1 < N; ++c) is_live = is_live || live_last.count(A[i][c]) > 0;
        PropSet P = 0;   // Eq. 1
        if (is_const) P = lattice_join(P, kConst);
        if (is_in) P = lattice_join(P, kIn);
        if (local_in || local_out) P = lattice_join(P, kLocal);
        if (is_live) P = lattice_join(P, kLive);
        if (is_out) P = lattice_join(P, kOut);
        C.P[i] = P;
        C.partner[i] = local_in ? rp[i] : (local_out ? wp[i] : -1);
    }
    C.match = true;   // Eq. 2
    for (int i = 0; i < M; ++i) C.match = C.match && C.P[i] != kTop;
    for (int i = 0; i < M; ++i)   // Eq. 3
        C.grouped[i] = (C.P[i] & kLive) || (!(C.P[i] & kLocal) && !(C.P[i] & kConst));
    return C;
}

// ===================================================================== rewrite
namespace {

int max_var(const std::vector<Stmt> &body) {
    int m = -1;
    for (const Stmt &s : body)
        if (s.kind == Stmt::kLoop) m = std::max({m, s.var, max_var(s.body)});
    return m;
}

Ref map_ref(const Ref &r, const std::vector<int> &to_buffer, const std::vector<bool> &grouped,
            int nvar) {
    Ref o = r;
    if (r.base != Ref::kParam) return o;
    if (to_buffer[r.id] >= 0) {        // rule 6: a Local parameter -> its buffer
        o.base = Ref::kBuffer;
        o.id = to_buffer[r.id];
    } else if (grouped[r.id]) {        // rule 6: a grouped parameter -> p[n]
        o.group_var = nvar;
    }
    return o;
}

ExprP map_expr(const ExprP &e, const std::vector<int> &to_buffer,
               const std::vector<bool> &grouped, int nvar) {
    if (e->op == Expr::kLeaf) return leaf(map_ref(e->ref, to_buffer, grouped, nvar));
    return node(e->op, map_expr(e->a, to_buffer, grouped, nvar),
                map_expr(e->b, to_buffer, grouped, nvar));
}

std::vector<Stmt> map_body(const std::vector<Stmt> &body, const std::vector<int> &to_buffer,
                           const std::vector<bool> &grouped, int nvar) {
    std::vector<Stmt> out;
    for (const Stmt &s : body) {
        Stmt t = s;
        if (s.kind == Stmt::kLoop) {
            t.body = map_body(s.body, to_buffer, grouped, nvar);
        } else {
            t.dst = map_ref(s.dst, to_buffer, grouped, nvar);
            t.rhs = map_expr(s.rhs, to_buffer, grouped, nvar);
        }
        out.push_back(t);
    }
    return out;
}

// With one buffer for the pair (in, out), would the body read rows of 'in'
// after it has written them through 'out'?  (A statement reads its right
// side before it writes, so a read in the writing statement itself is safe.)
bool needs_double_buffer(const Kernel &k, int in, int out) {
    const std::vector<Access> acc = accesses(k);
    std::vector<char> written(k.params[in].rows, 0);
    int cur = -1;
    std::vector<std::pair<int, int>> pending;   // writes of the current statement
    for (const Access &a : acc) {
        if (a.seq != cur) {
            for (auto &w : pending)
                for (int r = w.first; r < w.second; ++r) written[r] = 1;
            pending.clear();
            cur = a.seq;
        }
        if (a.write && a.param == out) pending.push_back({a.lo, a.hi});
        if (!a.write && a.param == in)
            for (int r = a.lo; r < a.hi; ++r)
                if (written[r]) return true;
    }
    return false;
}

Ref buffer_ref(int id) {
    Ref r;
    r.base = Ref::kBuffer;
    r.id = id;
    return r;
}

}  // namespace

Rewrite rewrite(const Program &prog, const Candidate &c) {
    if (!c.match) throw std::invalid_argument("rewrite: the calls do not match");
    const Kernel &k = prog.kernels[prog.calls[c.first].kernel];
    const int M = (int)k.params.size(), N = c.count;
    const int nvar = max_var(k.body) + 1;   // the loop over the calls
    Rewrite rw;
    Kernel &o = rw.kernel;
    o.name = k.name + "'";                  // rule 1
    o.params = k.params;
    o.locals = k.locals;
    o.group.assign(M, 0);
    for (int i = 0; i < M; ++i)             // rule 2
        if (c.grouped[i]) o.group[i] = N;

    // rules 3-4: one on-chip buffer per chained pair, initialised from the
    // pair's input; two when the body would overwrite rows it still reads
    std::vector<int> in_buf(M, -1), out_buf(M, -1);
    std::vector<Stmt> pre, post_iter, post;
    for (int i = 0; i < M; ++i) {
        if (c.P[i] != (kIn | kLocal)) continue;
        const int j = c.partner[i];
        const bool dbl = needs_double_buffer(k, i, j);
        const int b0 = (int)o.buffers.size();
        o.buffers.push_back({"buf" + std::to_string(b0), k.params[i].rows, k.params[i].cols});
        int b1 = b0;
        if (dbl) {
            b1 = (int)o.buffers.size();
            o.buffers.push_back({"buf" + std::to_string(b1), k.params[i].rows, k.params[i].cols});
        }
        in_buf[i] = b0;
        out_buf[j] = b1;
        rw.buffers.push_back({i, j, dbl});
        pre.push_back(assign(buffer_ref(b0), leaf(param(i))));
        if (dbl) post_iter.push_back(assign(buffer_ref(b0), leaf(buffer_ref(b1))));
        Ref pj = param(j);
        if (c.P[j] == (kLocal | kLive | kOut)) {          // rules 7-8
            pj.group_var = nvar;
            post_iter.push_back(assign(pj, leaf(buffer_ref(b1))));
            rw.stores_each_iteration.push_back(j);
        } else if (c.P[j] == (kLocal | kOut)) {           // rules 9-10
            post.push_back(assign(pj, leaf(buffer_ref(b1))));
            rw.stores_at_end.push_back(j);
        }
    }
    std::vector<int> to_buffer(M, -1);
    for (int i = 0; i < M; ++i) to_buffer[i] = in_buf[i] >= 0 ? in_buf[i] : out_buf[i];

    // rules 1 and 5: the loop over the calls around the mapped body
    std::vector<Stmt> body = map_body(k.body, to_buffer, c.grouped, nvar);
    body.insert(body.end(), post_iter.begin(), post_iter.end());
    o.body = pre;
    o.body.push_back(loop(nvar, 0, N, 1, body));
    o.body.insert(o.body.end(), post.begin(), post.end());

    // the collapsed call: Const -> the unique argument, {In,Local} -> the
    // first, {Local,Out} -> the last, grouped -> all of them
    rw.call.kernel = -1;   // set by the caller when the kernel is added
    rw.call.args.resize(M);
    for (int i = 0; i < M; ++i) {
        std::vector<int> all;
        for (int n = 0; n < N; ++n) all.push_back(prog.calls[c.first + n].args[i][0]);
        if (c.grouped[i]) rw.call.args[i] = all;
        else if (c.P[i] == (kLocal | kOut)) rw.call.args[i] = {all.back()};
        else rw.call.args[i] = {all.front()};
    }
    return rw;
}

Program kernel_looping_pass(const Program &prog, PassReport *report) {
    const std::vector<std::set<int>> LA = live_after(prog);
    Program out;
    out.tensors = prog.tensors;
    out.kernels = prog.kernels;
    out.outputs = prog.outputs;
    const int n = (int)prog.calls.size();
    auto single_args = [&](int c) {
        for (const auto &a : prog.calls[c].args)
            if (a.size() != 1) return false;
        return true;
    };
    int i = 0;
    while (i < n) {
        int run = i;   // the contiguous calls to the same kernel from i
        while (run + 1 < n && prog.calls[run + 1].kernel == prog.calls[i].kernel &&
               single_args(run + 1))
            ++run;
        int best = -1;
        Candidate cand;
        if (single_args(i))
            for (int e = run; e > i && best < 0; --e) {
                Candidate cd = analyse(prog, i, e - i + 1, LA[e]);
                if (cd.match) best = e, cand = cd;
            }
        if (best < 0) {
            out.calls.push_back(prog.calls[i]);
            ++i;
            continue;
        }
        Rewrite rw = rewrite(prog, cand);
        rw.call.kernel = (int)out.kernels.size();
        out.kernels.push_back(rw.kernel);
        out.calls.push_back(rw.call);
        if (report) {
            report->collapsed.push_back(cand);
            report->rewrites.push_back(rw);
        }
        i = best + 1;
    }
    return out;
}

// ===================================================================== interpreter
namespace {

struct Mat {
    int r = 0, c = 0;
    std::vector<double> v;
};

struct Frame {
    const Program &prog;
    const Kernel &k;
    const Call &call;
    Memory &mem;
    std::vector<std::vector<double>> locals, buffers;
    Vars vars;
};

// storage, rows, cols of what a reference names (before slicing)
std::vector<double> &target(Frame &f, const Ref &r, int &rows, int &cols) {
    if (r.base == Ref::kLocalTensor) {
        rows = f.k.locals[r.id].rows;
        cols = f.k.locals[r.id].cols;
        return f.locals[r.id];
    }
    if (r.base == Ref::kBuffer) {
        rows = f.k.buffers[r.id].rows;
        cols = f.k.buffers[r.id].cols;
        return f.buffers[r.id];
    }
    const std::vector<int> &args = f.call.args[r.id];
    int t;
    if (r.group_var >= 0) {
        const int n = var_value(f.vars, r.group_var);
        if (n < 0 || n >= (int)args.size()) throw std::runtime_error("group index out of range");
        t = args[n];
    } else {
        if (args.size() != 1) throw std::runtime_error("grouped parameter used without [n]");
        t = args[0];
    }
    rows = f.prog.tensors[t].rows;
    cols = f.prog.tensors[t].cols;
    if (rows != f.k.params[r.id].rows || cols != f.k.params[r.id].cols)
        throw std::runtime_error("argument shape differs from the parameter's");
    return f.mem[t];
}

Mat read(Frame &f, const Ref &r) {
    int rows, cols;
    const std::vector<double> &d = target(f, r, rows, cols);
    const auto rr = ref_rows(r, rows, f.vars);
    Mat m;
    m.r = rr.second - rr.first;
    m.c = cols;
    m.v.assign(d.begin() + (size_t)rr.first * cols, d.begin() + (size_t)rr.second * cols);
    return m;
}

Mat eval(Frame &f, const Expr &e) {
    if (e.op == Expr::kLeaf) return read(f, e.ref);
    const Mat a = eval(f, *e.a), b = eval(f, *e.b);
    Mat o;
    if (e.op == Expr::kMatMul) {
        if (a.c != b.r) throw std::runtime_error("matmul shape mismatch");
        o.r = a.r;
        o.c = b.c;
        o.v.assign((size_t)o.r * o.c, 0.0);
        for (int i = 0; i < a.r; ++i)
            for (int j = 0; j < b.c; ++j) {
                double s = 0.0;
                for (int t = 0; t < a.c; ++t) s += a.v[(size_t)i * a.c + t] * b.v[(size_t)t * b.c + j];
                o.v[(size_t)i * o.c + j] = s;
            }
        return o;
    }
    if (a.r != b.r || a.c != b.c) throw std::runtime_error("elementwise shape mismatch");
    o = a;
    for (size_t i = 0; i < o.v.size(); ++i)
        o.v[i] = e.op == Expr::kAdd ? a.v[i] + b.v[i]
               : e.op == Expr::kSub ? a.v[i] - b.v[i] : a.v[i] * b.v[i];
    return o;
}

void exec(Frame &f, const std::vector<Stmt> &body) {
    for (const Stmt &s : body) {
        if (s.kind == Stmt::kLoop) {
            for (int i = s.lo; i < s.hi; i += s.step) {
                f.vars[s.var] = i;
                exec(f, s.body);
            }
            f.vars.erase(s.var);
            continue;
        }
        const Mat m = eval(f, *s.rhs);   // value semantics: the right side first
        int rows, cols;
        std::vector<double> &d = target(f, s.dst, rows, cols);
        const auto rr = ref_rows(s.dst, rows, f.vars);
        if (m.r != rr.second - rr.first || m.c != cols)
            throw std::runtime_error("assignment shape mismatch");
        for (size_t i = 0; i < m.v.size(); ++i) {
            double &x = d[(size_t)rr.first * cols + i];
            x = s.kind == Stmt::kAccumulate ? x + m.v[i] : m.v[i];
        }
    }
}

}  // namespace

Memory run_program(const Program &prog, const Memory &init) {
    Memory mem = init;
    for (size_t t = 0; t < prog.tensors.size(); ++t)
        if (mem[t].size() != (size_t)prog.tensors[t].rows * prog.tensors[t].cols)
            throw std::runtime_error("initial memory does not match the tensors");
    for (const Call &call : prog.calls) {
        const Kernel &k = prog.kernels[call.kernel];
        if (call.args.size() != k.params.size()) throw std::runtime_error("argument count");
        Frame f{prog, k, call, mem, {}, {}, {}};
        for (const Tensor &t : k.locals) f.locals.emplace_back((size_t)t.rows * t.cols, 0.0);
        for (const Tensor &t : k.buffers) f.buffers.emplace_back((size_t)t.rows * t.cols, 0.0);
        exec(f, k.body);
    }
    return mem;
}

// ===================================================================== printing
namespace {

std::string var_name(int v, int nvar) { return v == nvar ? "n" : std::string(1, (char)('t' + v)); }

std::string shape(const Tensor &t, int group) {
    std::ostringstream s;
    s << "[";
    if (group) s << group << "x";
    s << t.rows << "x" << t.cols << "]";
    return s.str();
}

std::string ref_str(const Kernel &k, const Ref &r, int nvar) {
    std::string s = r.base == Ref::kParam ? k.params[r.id].name
                  : r.base == Ref::kLocalTensor ? k.locals[r.id].name : k.buffers[r.id].name;
    if (r.group_var >= 0) s += "[" + var_name(r.group_var, nvar) + "]";
    if (r.sliced) {
        std::string lo = std::to_string(r.lo_const);
        if (r.lo_var >= 0) {
            const std::string v = (r.lo_step == 1 ? "" : std::to_string(r.lo_step) + "*") +
                                  var_name(r.lo_var, nvar);
            lo = r.lo_const ? lo + "+" + v : v;
        }
        s += "[" + lo + "::" + lo + "+" + std::to_string(r.len) + "]";
    }
    return s;
}

std::string expr_str(const Kernel &k, const Expr &e, int nvar) {
    if (e.op == Expr::kLeaf) return ref_str(k, e.ref, nvar);
    const char *op = e.op == Expr::kAdd ? " + " : e.op == Expr::kSub ? " - "
                   : e.op == Expr::kEMul ? " .* " : " * ";
    auto sub = [&](const Expr &x) {
        const std::string t = expr_str(k, x, nvar);
        return x.op == Expr::kLeaf ? t : "(" + t + ")";
    };
    return sub(*e.a) + op + sub(*e.b);
}

void body_str(const Kernel &k, const std::vector<Stmt> &body, int indent, int nvar,
              std::ostringstream &o) {
    const std::string pad(indent, ' ');
    for (const Stmt &s : body) {
        if (s.kind == Stmt::kLoop) {
            const std::string v = var_name(s.var, nvar);
            o << pad << "for (" << v << " = " << s.lo << "; " << v << " < " << s.hi << "; " << v
              << " += " << s.step << ")\n";
            body_str(k, s.body, indent + 2, nvar, o);
        } else {
            o << pad << ref_str(k, s.dst, nvar) << (s.kind == Stmt::kAccumulate ? " += " : " = ")
              << expr_str(k, *s.rhs, nvar) << "\n";
        }
    }
}

}  // namespace

std::string print_kernel(const Kernel &k) {
    std::ostringstream o;
    o << k.name << "(";
    for (size_t i = 0; i < k.params.size(); ++i)
        o << (i ? ", " : "") << k.params[i].name
          << shape(k.params[i], k.group.empty() ? 0 : k.group[i]);
    o << ")\n";
    for (const Tensor &t : k.buffers) o << "  @onchip " << t.name << shape(t, 0) << "\n";
    // (the loop over the calls, the outermost loop of a looped kernel, prints as n)
    body_str(k, k.body, 2, k.group.empty() ? -1 : max_var(k.body), o);
    return o.str();
}

std::string print_call(const Program &prog, const Call &c) {
    std::ostringstream o;
    o << prog.kernels[c.kernel].name << "(";
    for (size_t i = 0; i < c.args.size(); ++i) {
        o << (i ? ", " : "");
        if (c.args[i].size() == 1 && (prog.kernels[c.kernel].group.empty() ||
                                      prog.kernels[c.kernel].group[i] == 0)) {
            o << prog.tensors[c.args[i][0]].name;
        } else {
            o << "{";
            for (size_t j = 0; j < c.args[i].size(); ++j)
                o << (j ? "," : "") << prog.tensors[c.args[i][j]].name;
            o << "}";
        }
    }
    o << ")";
    return o.str();
}

}  // namespace klp
