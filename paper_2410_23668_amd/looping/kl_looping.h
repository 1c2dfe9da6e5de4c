// Kernel looping as a compiler pass (Sec. 3) over a small kernel-call IR,
// with an interpreter that runs a program before and after the rewrite.
//
// The IR: a program declares 2-D tensors (rows x cols, doubles) and makes a
// straight-line list of calls; a kernel has tensor parameters, private local
// tensors and a body of statements (assignment with value semantics,
// accumulation, counted loops) over expressions (elementwise add, subtract,
// multiply, and matrix product) of tensor references, each optionally a row
// slice [lo + step * v, + len) of a loop variable v.
//
// The pass follows Sec. 3.1 and 3.2:
//   - usage analysis of a kernel body (Reads, Writes, ReadSpace, WriteSpace
//     per parameter, by running the loops over row sets) and liveness over the
//     call list (LiveAfter of each call);
//   - the usage properties of each parameter over a candidate list of calls
//     (Fig. 6a: Const, In, Local, Live, Out), joined on the lattice of
//     Fig. 6b into P(p) (Eq. 1); Match (Eq. 2) holds when no P(p) is the top;
//   - the rewrite (Fig. 7, rules 1-10): one looped kernel with the grouped
//     parameters (Eq. 3) given an outer dimension N, each chained pair of
//     Local parameters turned into an on-chip buffer (double-buffered where
//     the body would overwrite rows it still reads), stores of the buffers
//     each iteration (Local, Live, Out) or once at the end (Local, Out), and
//     the calls collapsed into one call whose grouped arguments are lists;
//   - a greedy driver that collapses the longest matching run of contiguous
//     calls to one kernel, then moves on (Sec. 3.1, last paragraph).
//
// Host code only (C++17); no GPU involved.
#pragma once

#include <map>
#include <memory>
#include <set>
#include <string>
#include <vector>

namespace klp {

// ------------------------------------------------------------ usage properties
enum Prop : unsigned { kConst = 1u, kIn = 2u, kLocal = 4u, kLive = 8u, kOut = 16u };
using PropSet = unsigned;              // an OR of Prop bits
constexpr PropSet kTop = 1u << 5;      // the lattice's top: a match failure

// Join on the lattice of Fig. 6b: the least element above both (computed on
// the lattice's Hasse diagram), kTop when it is the top.
PropSet lattice_join(PropSet a, PropSet b);
// The lattice's elements below the top: the empty set, the five singletons and
// the seven pairs/triples (1)-(7) of Fig. 6b.
const std::vector<PropSet> &lattice_elements();
std::string prop_string(PropSet p);    // e.g. "{In,Local}", "T" for the top

// ------------------------------------------------------------------------- IR
struct Tensor {
    std::string name;
    int rows = 1, cols = 1;
};

struct Ref {
    enum Base { kParam, kLocalTensor, kBuffer } base = kParam;
    int id = 0;                 // parameter, local or buffer index
    int group_var = -1;         // loop variable selecting the group member p[n], or -1
    bool sliced = false;        // rows [lo_const + lo_step * var(lo_var), + len)
    int lo_const = 0, lo_var = -1, lo_step = 0, len = 0;
};

struct Expr {
    enum Op { kLeaf, kAdd, kSub, kEMul, kMatMul } op = kLeaf;
    Ref ref;                                   // kLeaf
    std::shared_ptr<const Expr> a, b;          // operands
};
using ExprP = std::shared_ptr<const Expr>;

struct Stmt {
    enum Kind { kAssign, kAccumulate, kLoop } kind = kAssign;
    Ref dst;                    // kAssign (dst = rhs), kAccumulate (dst += rhs)
    ExprP rhs;
    int var = 0, lo = 0, hi = 0, step = 1;     // kLoop: for (var = lo; var < hi; var += step)
    std::vector<Stmt> body;
};

// Calls pass distinct tensors to a kernel's parameters (no aliasing within a
// call), and a body assigns a local before reading it.
struct Kernel {
    std::string name;
    std::vector<Tensor> params;
    std::vector<int> group;     // looped kernels: per parameter, N when grouped ([N x S]), else 0
    std::vector<Tensor> locals; // kernel-private tensors (off-chip temporaries)
    std::vector<Tensor> buffers;// on-chip buffers introduced by the rewrite
    std::vector<Stmt> body;
};

struct Call {
    int kernel = 0;
    std::vector<std::vector<int>> args;   // per parameter: one tensor, or the group's tensors
};

struct Program {
    std::vector<Tensor> tensors;
    std::vector<Kernel> kernels;
    std::vector<Call> calls;
    std::set<int> outputs;      // tensors live at the end of the program
};

// Builders for kernel bodies.
Ref param(int id);
Ref local(int id);
Ref rows(Ref r, int lo_const, int lo_var, int lo_step, int len);
ExprP leaf(const Ref &r);
ExprP add(ExprP a, ExprP b);
ExprP sub(ExprP a, ExprP b);
ExprP emul(ExprP a, ExprP b);
ExprP matmul(ExprP a, ExprP b);
Stmt assign(const Ref &dst, ExprP rhs);
Stmt accumulate(const Ref &dst, ExprP rhs);
Stmt loop(int var, int lo, int hi, int step, std::vector<Stmt> body);

// ------------------------------------------------------------------- analysis
struct Usage {                  // per parameter of a kernel
    std::vector<std::set<int>> read_rows, write_rows;   // ReadSpace / WriteSpace (rows)
    bool reads(int p) const { return !read_rows[p].empty(); }
    bool writes(int p) const { return !write_rows[p].empty(); }
};
Usage usage_of(const Kernel &k);

// LiveAfter(c) for every call: the tensors a later call reads before it
// overwrites them whole, or that the program outputs.
std::vector<std::set<int>> live_after(const Program &prog);

struct Candidate {
    int first = 0, count = 0;   // calls first .. first + count - 1
    std::vector<PropSet> P;     // P(p_i), Eq. 1
    std::vector<int> partner;   // Local parameters: the other parameter of the pair, else -1
    std::vector<bool> grouped;  // Group(p_i), Eq. 3
    bool match = false;         // Match(C), Eq. 2
};

// Usage properties of the calls first .. first + count - 1 (all to one
// kernel, count >= 2) with the given LiveAfter of the last of them.
Candidate analyse(const Program &prog, int first, int count, const std::set<int> &live_last);

// --------------------------------------------------------------- rewrite
struct Rewrite {
    Kernel kernel;              // the looped kernel
    Call call;                  // the collapsed call
    struct Buffer {
        int in_param, out_param;
        bool double_buffered;
    };
    std::vector<Buffer> buffers;
    std::vector<int> stores_each_iteration;   // rule 8
    std::vector<int> stores_at_end;           // rule 10
};
Rewrite rewrite(const Program &prog, const Candidate &c);

struct PassReport {
    std::vector<Candidate> collapsed;
    std::vector<Rewrite> rewrites;
};
// The greedy driver: from each call, the longest run of contiguous calls to
// the same kernel that matches (two calls or more) is collapsed.
Program kernel_looping_pass(const Program &prog, PassReport *report);

// ---------------------------------------------------------------- interpreter
using Memory = std::vector<std::vector<double>>;   // per program tensor, row-major
Memory run_program(const Program &prog, const Memory &init);

// Printing in the notation of the paper's examples.
std::string print_kernel(const Kernel &k);
std::string print_call(const Program &prog, const Call &c);

}  // namespace klp
