// Host runtime behind the C ABI in include/kl.h: argument validation, the
// packed weight arena, the RoPE table, step scratch and the launch plans of
// the three schedules.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "kl.h"
#include "kl_internal.h"

using namespace kl;

struct kl_state {
    kl_config cfg;
    int device;
    int Hp, Ap, Fp, qkv_rg, o_rg, gu_rg, down_rg, head_rg;
    size_t layer_stride, off_attn_norm, off_ffn_norm, off_qkv, off_o, off_gu, off_down;
    size_t off_qkv_bias;
    size_t off_router, gu_estride, down_estride;   // mixture of experts
    size_t off_final_norm, off_lm_head, off_embed;
    uint8_t *arena;
    size_t arena_bytes;
    float2 *rope;
    uint8_t *scratch;                 // step scratch laid out by plan_scratch(max_batch)
    size_t scratch_bytes;
    uint8_t *static_scratch;          // this device's address of the library's static scratch
    int KSo, KSd, KSg, KSq;           // K slices of the batched O, down, gate/up, q/k/v products
    int Sg, Sc, Rc, KTc;
    int *err;                         // device error word (its own allocation, 256 B)
    unsigned *epoch;                  // first tag of the next step (in the same allocation)
    unsigned long long *keys;         // argmax keys of the token loop: [2][max_batch]
    // the per-layer schedule as a graph, for the caller buffers it was built on
    hipGraph_t graph;
    hipGraphExec_t graph_exec;
    const void *graph_key[10];
    size_t off_dummy;                 // arena offset of a zero tile (the load rings' spare loads)
    unsigned long long *trace;
    int trace_max;
    int32_t *rowmaps;                 // device row maps used by set_layer / set_globals
    const int32_t *maps[5];           // by RowMap
    int nwg, lds_bytes;
    int lds_red, lds_sm, lds_bar;
    int lds_red_seq;                  // the GEMV partial sums on the per-sequence path
    bool multi_ok;                    // up to kMultiSeq sequences share a GEMV pass
    int batched_from;                 // first batch of the matrix-core path
};

namespace {

thread_local std::string g_last_error;

kl_status fail(kl_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

#define HIP_TRY(expr)                                                                      \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return fail(e_ == hipErrorOutOfMemory ? KL_ERR_OUT_OF_MEMORY : KL_ERR_HIP,     \
                        "%s failed: %s", #expr, hipGetErrorString(e_));                    \
    } while (0)

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

kl_status validate_config(const kl_config *c) {
    if (!c) return fail(KL_ERR_INVALID_ARGUMENT, "config is NULL");
    if (c->n_layers < 1 || c->hidden < 1 || c->n_heads < 1 || c->n_kv_heads < 1 ||
        c->head_dim < 1 || c->ffn_dim < 1 || c->vocab < 1 || c->max_batch < 1 || c->max_seq < 1)
        return fail(KL_ERR_INVALID_ARGUMENT, "every config dimension must be >= 1");
    if (!(c->rms_eps > 0.f) || !std::isfinite(c->rms_eps))
        return fail(KL_ERR_INVALID_ARGUMENT, "rms_eps must be a positive finite number");
    if (!(c->rope_theta > 1.f) || !std::isfinite(c->rope_theta))
        return fail(KL_ERR_INVALID_ARGUMENT, "rope_theta must be a finite number > 1");
    if (c->head_dim != 64 && c->head_dim != 128)
        return fail(KL_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", c->head_dim);
    if (c->n_heads % c->n_kv_heads != 0)
        return fail(KL_ERR_UNSUPPORTED, "n_heads %d is not a multiple of n_kv_heads %d",
                    c->n_heads, c->n_kv_heads);
    const int g = c->n_heads / c->n_kv_heads;
    if (g != 1 && g != 2 && g != 4 && g != 8 && !(g == 3 && c->head_dim == 128))
        return fail(KL_ERR_UNSUPPORTED, "query heads per KV head must be 1, 2, 4 or 8, or 3 with "
                                        "head_dim 128 (got %d)", g);
    if (c->qkv_bias != 0 && c->qkv_bias != 1)
        return fail(KL_ERR_INVALID_ARGUMENT, "qkv_bias must be 0 or 1");
    if (c->n_experts < 0 || c->n_experts > 8)   // (the router is one packed row group)
        return fail(KL_ERR_UNSUPPORTED, "n_experts %d outside [0, 8]", c->n_experts);
    if (c->n_experts > 1 && (c->top_k < 1 || c->top_k > 2 || c->top_k > c->n_experts))
        return fail(KL_ERR_UNSUPPORTED, "top_k %d unsupported with %d experts (1 or 2)",
                    c->top_k, c->n_experts);
    if (c->hidden % 8 != 0 || c->ffn_dim % 8 != 0)
        return fail(KL_ERR_UNSUPPORTED, "hidden and ffn_dim must be multiples of 8");
    if (c->max_batch > 4096) return fail(KL_ERR_UNSUPPORTED, "max_batch above 4096");
    if ((int64_t)c->vocab >= (1 << 28) || (int64_t)c->ffn_dim >= (1 << 27))
        return fail(KL_ERR_UNSUPPORTED, "vocab or ffn_dim too large");
    return KL_OK;
}

// FFN column blocks: the largest divisor of the k-tile count of ffn_dim that
// is at most 32 (and at most the grid).
int largest_divisor_at_most(int n, int cap) {
    for (int k = std::min(n, cap); k > 1; --k)
        if (n % k == 0) return k;
    return 1;
}

// K slices of a batched product over n K units of t k-tiles each, for a
// matrix of nblk 16-row blocks: the fewest slices (a divisor of n, at most
// kMaxKSlices) whose K range stays resident in LDS and that give every
// workgroup kWaves blocks or more; failing that, the resident choice with the
// most blocks per workgroup; if no slice fits in LDS, the most slices (the
// activations then stream through LDS in chunks).
int batched_k_slices(int n, int t, int nblk, int nwg) {
    int best = -1;
    for (int s = 1; s <= std::min(n, kMaxKSlices); ++s) {
        if (n % s || (n / s) * t * kTileK > kGemmResidentK) continue;
        best = s;
        if ((long long)nblk * s >= (long long)kWaves * nwg) break;
    }
    return best > 0 ? best : largest_divisor_at_most(n, kMaxKSlices);
}
// K slices of the gate/up and q/k/v products, whose K-slice partial sums a
// grid-wide fold reads back (the SwiGLU fold, the q/k/v fold): the fewest
// slices (a divisor of n, at most kMaxKSlices) whose K range is at most two
// resident ranges (the activations then stream through LDS) and that give
// every workgroup kWaves / 2 blocks or more; failing that, batched_k_slices.
// Fewer slices halve what the fold reads.  (8B shape, batch 32: 7.95 ms with
// 4 gate/up and 8 q/k/v slices, 7.48 with 2 and 4; the same for the O and
// down products, whose partials the next RMSNorm folds, gained nothing.)
int folded_k_slices(int n, int t, int nblk, int nwg) {
    for (int s = 1; s <= std::min(n, kMaxKSlices); ++s) {
        if (n % s || (n / s) * t * kTileK > 2 * kGemmResidentK) continue;
        if ((long long)nblk * s >= (long long)(kWaves / 2) * nwg) return s;
    }
    return batched_k_slices(n, t, nblk, nwg);
}

// Dynamic LDS layout of the step kernel (offsets in floats): the activation
// vector / attention area, the GEMV wave partials, 64 floats of small
// reductions and flags, then the barrier bases.
void lds_layout_for(kl_state &s) {
    const kl_config &c = s.cfg;
    const int g = c.n_heads / c.n_kv_heads, d = c.head_dim;
    // attention: the queries, the new key and value, and (streaming item)
    // the waves' (max, sum, output) per head of their team or (short-chunk
    // item) a sub-chunk's scores, the softmax state and the waves' outputs
    const int hg = std::min(g, 4);
    const int sub = kWaves * kAttnLoads * (64 / (d / 8));
    // (+ the streaming item's per-wave score tiles, 16 x 16 floats)
    const int attn_main = std::max(g * d + 2 * kWaves * hg + kWaves * hg * d + d + kWaves * 256,
                                   g * d + g * sub + g * 4 + kWaves * g * d + d);
    // O projection: o, chunk weights, running sums, the chunk results
    const int oproj_stage = d + kMergeChunks + 4 + kMergeChunks * (d + 2);
    const auto round64 = [](int v) { return (v + 63) & ~63; };
    const int rs = kWaves * kRgBatch * kTileRows;   // one sequence's GEMV partial sums
    // per-sequence path, one sequence per GEMV pass: activations and RoPE row
    const int one = round64(std::max({2 * s.Hp + d, s.KTc * kTileK, attn_main, oproj_stage}));
    // kMultiSeq sequences per pass: their activations and RoPE rows, their
    // SwiGLU blocks, their merged attention outputs before the merge's area
    const int multi = round64(std::max({kMultiSeq * (s.Hp + d), kMultiSeq * s.KTc * kTileK,
                                        kMultiSeq * d + kMergeChunks + 4 + kMergeChunks * (d + 2),
                                        attn_main, 2 * s.Hp + d}));
    // The first batch of the matrix-core path: with several sequences per
    // GEMV pass the per-sequence path serves up to kMultiSeq sequences (a
    // mixture of experts: up to kMfmaBatch - 1, as its routing needs).  The
    // matrix-core path's area (and its partial sums after it) may overlap
    // the per-sequence path's partial sums: a launch runs one of the two.
    const auto layout = [&](bool mu) {
        s.multi_ok = mu;
        s.batched_from = c.n_experts > 1 ? kMfmaBatch : (mu ? kMultiSeq + 1 : kBatchedFrom);
        const int seq_a = mu ? multi : one;
        const int seq_end = seq_a + (mu ? kMultiSeq : 1) * rs;
        const bool bat = c.max_batch >= s.batched_from;
        const int bat_a = bat ? round64(std::max(seq_a, kGemmLdsBytes / 4)) : seq_a;
        s.lds_red_seq = seq_a;
        s.lds_red = bat_a;
        s.lds_sm = std::max(seq_end, bat_a + rs);
        s.lds_bar = s.lds_sm + 64;
        // + the step's epoch, position and validity per sequence, the head's
        // argmax keys of a group of sequences, the experts and their weights
        // per sequence (two slots)
        s.lds_bytes = (s.lds_bar + 2 * kBarGroups + 4 + 2 * kMfmaBatch + 2 * kGemmBatch +
                       4 * kMfmaBatch) * (int)sizeof(float);
    };
    layout(c.max_batch >= 2);
    if (s.multi_ok && s.lds_bytes > 160 * 1024 - 256) layout(false);
}

// Step scratch for a batch of B sequences (byte offsets from its base; every
// region 256-byte aligned):
//   grid barrier counters (16 groups, 256 B apart) and the local counters:
//     qkv and attention per KV head, gate/up per FFN column block, and at
//     matrix-core steps the batched RMSNorm slice counters (256 bytes apart);
//   the residual stream, int64 fixed point [B][Hp];
//   the per-sequence path's tagged words (8 bytes each, for up to
//     kMfmaBatch - 1 sequences): rotated queries [B][nq d], the new key and
//     value [B][nkv][d], chunk results [B][nkv][group][C][d + 2], the SwiGLU
//     output [B][Fp];
//   the matrix-core path's rotated queries [B][nq d] and attention chunk
//     partials: outputs [B nkv C][group][d], (max, sum) pairs;
//   the matrix-core path's two-term bf16 activations (both terms, [B][Hp],
//     [B][Fp], [B][nq d]);
//   on the matrix-core path also: the second residual buffer, the fp32 K-slice
//     partials of the O and down projections [slices][B][Hp] and of the
//     gate/up or q/k/v product (never live at the same time), and the
//     RMSNorm sums of squares per kGemmChunkK columns [B][slices].
struct ScratchPlan {
    int B;
    bool batched;
    size_t off_bar, off_cnt, off_cnt_end;
    size_t off_x, off_q, off_po, off_ps, off_act, off_actm, off_acto;
    size_t off_qll, off_kvll, off_poll, off_mll;
    size_t off_x2, off_xp, off_gp, off_ss;
    size_t total;
};

ScratchPlan plan_scratch(const kl_state &S, int B) {
    const kl_config &c = S.cfg;
    const int d = c.head_dim, g = c.n_heads / c.n_kv_heads, nkv = c.n_kv_heads;
    ScratchPlan p{};
    p.B = B;
    p.batched = B >= S.batched_from;
    size_t so = 0;
    auto take = [&](size_t bytes) {
        const size_t o = so;
        so = align_up(so + bytes, 256);
        return o;
    };
    const int nslices = (S.Hp + kGemmChunkK - 1) / kGemmChunkK;
    const int norm_cnts = p.batched ? kNormCntStride * nslices : 0;
    p.off_bar = take(kBarBytes);
    p.off_cnt = take((size_t)(2 * nkv + S.Sc + norm_cnts) * 4);
    p.off_cnt_end = so;
    const size_t items = (size_t)nkv * std::max(B, S.Sg);   // >= B * nkv * C for this batch
    p.off_x = take((size_t)B * S.Hp * 8);
    const int bl = std::min(B, S.batched_from - 1);           // per-sequence steps
    const size_t items_ll = (size_t)nkv * std::max(bl, S.Sg);
    p.off_qll = take((size_t)bl * c.n_heads * d * 8);
    p.off_kvll = take((size_t)bl * nkv * d * 8);
    p.off_poll = take(items_ll * g * (d + 2) * 8);
    const int topk = c.n_experts > 1 ? c.top_k : 1;          // expert slots per token
    p.off_mll = take((size_t)bl * topk * S.Fp * 8);
    p.off_q = take((size_t)B * c.n_heads * d * 4);
    p.off_po = take(items * g * d * 4);
    p.off_ps = take(items * g * 2 * 4);
    p.off_act = take((size_t)B * S.Hp * 2 * 2);
    p.off_actm = take((size_t)B * S.Fp * 2 * 2);
    p.off_acto = take((size_t)B * S.Ap * 2 * 2);
    if (p.batched) {
        const size_t qkv_rows = (size_t)nkv * S.qkv_rg * kTileRows;
        p.off_x2 = take((size_t)B * S.Hp * 8);
        p.off_xp = take((size_t)std::max(S.KSo, S.KSd) * B * S.Hp * 4);
        p.off_gp = take(std::max((size_t)S.KSg * B * S.gu_rg * kTileRows,
                                 (size_t)S.KSq * B * qkv_rows) * 4);
        p.off_ss = take((size_t)B * nslices * 4);
    }
    p.total = so;
    return p;
}

// Points the step's scratch fields at the regions of 'plan' inside 'base'.
void bind_scratch(StepParams &P, uint8_t *base, const ScratchPlan &p, const kl_state &S) {
    const int B = p.B;
    P.bar = reinterpret_cast<unsigned long long *>(base + p.off_bar);
    P.cnt = reinterpret_cast<unsigned *>(base + p.off_cnt);
    P.xf = reinterpret_cast<long long *>(base + p.off_x);
    P.q = reinterpret_cast<float *>(base + p.off_q);
    P.q_ll = reinterpret_cast<unsigned long long *>(base + p.off_qll);
    P.kv_ll = reinterpret_cast<unsigned long long *>(base + p.off_kvll);
    P.po_ll = reinterpret_cast<unsigned long long *>(base + p.off_poll);
    P.m_ll = reinterpret_cast<unsigned long long *>(base + p.off_mll);
    P.part_o = reinterpret_cast<float *>(base + p.off_po);
    P.part_s = reinterpret_cast<float *>(base + p.off_ps);
    P.act = reinterpret_cast<uint16_t *>(base + p.off_act);
    P.act_lo = P.act + (size_t)B * S.Hp;
    P.actm = reinterpret_cast<uint16_t *>(base + p.off_actm);
    P.actm_lo = P.actm + (size_t)B * S.Fp;
    P.acto = reinterpret_cast<uint16_t *>(base + p.off_acto);
    P.acto_lo = P.acto + (size_t)B * S.Ap;
    P.xf2 = p.batched ? reinterpret_cast<long long *>(base + p.off_x2) : nullptr;
    P.xpart = p.batched ? reinterpret_cast<float *>(base + p.off_xp) : nullptr;
    P.gpart = p.batched ? reinterpret_cast<float *>(base + p.off_gp) : nullptr;
    P.ssp = p.batched ? reinterpret_cast<float *>(base + p.off_ss) : nullptr;
    P.xpart_stride = B * S.Hp;
    P.gpart_stride = B * S.gu_rg * kTileRows;
    P.qpart_stride = B * S.cfg.n_kv_heads * S.qkv_rg * kTileRows;
}

void free_state(kl_state *s) {
    if (!s) return;
    if (s->arena) (void)hipFree(s->arena);
    if (s->rope) (void)hipFree(s->rope);
    if (s->scratch) (void)hipFree(s->scratch);
    if (s->err) (void)hipFree(s->err);
    if (s->keys) (void)hipFree(s->keys);
    if (s->graph_exec) (void)hipGraphExecDestroy(s->graph_exec);
    if (s->graph) (void)hipGraphDestroy(s->graph);
    if (s->rowmaps) (void)hipFree(s->rowmaps);
    delete s;
}

// Whether the workgroups of one launch running 'phases' (a single phase, or
// several) wait for each other inside it; such a launch must be cooperative,
// so that the whole grid is resident.  Waits on work of an earlier launch are
// already satisfied when the launch starts (stream order), so only in-launch
// hand-offs count:
//   several phases in one launch      grid barriers and local counters;
//   matrix-core path, single phases:
//     qkv       its product's grid barrier before the fold, and the RMSNorm
//               slice counters;
//     oproj     with several attention chunks, the merge's grid barrier;
//     gateup    the RMSNorm slice counters;
//     down      the SwiGLU fold's grid barrier;
//     head      the final RMSNorm's slice counters;
//     attn      none (its counters were completed by the qkv launch);
//   per-sequence path, single phases: none (every counter a phase waits on
//   belongs to an earlier phase).
bool launch_waits_inside(int phases, bool batched, int C) {
    if (phases & kPhEmbed) return phases != kPhEmbed;
    if (__builtin_popcount((unsigned)phases) > 1) return true;
    if (!batched) return false;
    if (phases == kPhAttn) return false;
    if (phases == kPhOproj) return C > 1;
    return true;
}

StepParams base_params(const kl_state &s) {
    const kl_config &c = s.cfg;
    StepParams P{};
    P.L = c.n_layers; P.H = c.hidden; P.nq = c.n_heads; P.nkv = c.n_kv_heads; P.d = c.head_dim;
    P.F = c.ffn_dim; P.V = c.vocab; P.group = c.n_heads / c.n_kv_heads;
    P.Hp = s.Hp; P.Ap = s.Ap; P.Fp = s.Fp;
    P.qkv_rg = s.qkv_rg; P.o_rg = s.o_rg; P.gu_rg = s.gu_rg; P.down_rg = s.down_rg;
    P.head_rg = s.head_rg;
    P.Sg = s.Sg; P.Sc = s.Sc; P.Rc = s.Rc; P.KTc = s.KTc;
    P.eps = c.rms_eps; P.max_seq = c.max_seq;
    P.arena = s.arena; P.layer_stride = s.layer_stride;
    P.off_attn_norm = s.off_attn_norm; P.off_ffn_norm = s.off_ffn_norm; P.off_qkv = s.off_qkv;
    P.off_qkv_bias = s.off_qkv_bias; P.qkv_bias = c.qkv_bias ? 1 : 0;
    P.off_o = s.off_o; P.off_gu = s.off_gu; P.off_down = s.off_down;
    P.E = c.n_experts > 1 ? c.n_experts : 1; P.topk = c.n_experts > 1 ? c.top_k : 1;
    P.off_router = s.off_router; P.gu_estride = s.gu_estride; P.down_estride = s.down_estride;
    P.embed = reinterpret_cast<const uint16_t *>(s.arena + s.off_embed);
    P.final_norm = reinterpret_cast<const float *>(s.arena + s.off_final_norm);
    P.lm_head = reinterpret_cast<const uint16_t *>(s.arena + s.off_lm_head);
    P.rope = s.rope;
    P.KSo = s.KSo; P.KSd = s.KSd; P.KSg = s.KSg; P.KSq = s.KSq;
    P.err = s.err;
    P.epoch_ptr = s.epoch;
    P.dummy = s.arena + s.off_dummy;
    P.nwg = s.nwg;
    P.lds_red = s.lds_red; P.lds_sm = s.lds_sm; P.lds_bar = s.lds_bar;
    P.trace = s.trace;
    P.trace_max = s.trace_max;
    return P;
}

}  // namespace

extern "C" {

const char *kl_last_error(void) { return g_last_error.c_str(); }

size_t kl_kv_cache_bytes(const kl_config *cfg, int32_t batch, int32_t capacity) {
    if (!cfg || validate_config(cfg) != KL_OK || batch < 1 || capacity < 1) return 0;
    return (size_t)cfg->n_layers * batch * cfg->n_kv_heads * (size_t)capacity * cfg->head_dim *
           sizeof(uint16_t);
}

// Validates one layer's pointers.
kl_status check_layer_ptrs(const kl_layer_ptrs &L, int l, bool bias, bool moe) {
    const void *ps[] = {L.attn_norm, L.wq, L.wk, L.wv, L.wo, L.ffn_norm, L.w_gate, L.w_up,
                        L.w_down, L.bq, L.bk, L.bv, L.w_router};
    for (int i = 0; i < 13; ++i) {
        if ((i >= 9 && i < 12 && !bias) || (i == 12 && !moe)) continue;
        if (!ps[i])
            return fail(KL_ERR_INVALID_ARGUMENT, "layer %d has a NULL weight%s pointer", l,
                        i == 12 ? " (router)" : (i >= 9 ? " (bias)" : ""));
        if (!aligned(ps[i], 2))
            return fail(KL_ERR_INVALID_ARGUMENT, "layer %d weight not 2-byte aligned", l);
    }
    return KL_OK;
}

kl_status kl_model_create(const kl_config *cfg, kl_state **out) {
    g_last_error.clear();
    if (!out) return fail(KL_ERR_INVALID_ARGUMENT, "out is NULL");
    *out = nullptr;
    kl_status st = validate_config(cfg);
    if (st != KL_OK) return st;
    hipStream_t s = nullptr;

    kl_state *S = new kl_state();
    S->cfg = *cfg;
    const kl_config &c = S->cfg;
    auto bail = [&](kl_status code) { free_state(S); return code; };
#define TRY(expr)                                                                          \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return bail(fail(e_ == hipErrorOutOfMemory ? KL_ERR_OUT_OF_MEMORY : KL_ERR_HIP,  \
                             "%s failed: %s", #expr, hipGetErrorString(e_)));              \
    } while (0)

    TRY(hipGetDevice(&S->device));
    int ncu = 0, coop = 0;
    TRY(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, S->device));
    TRY(hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, S->device));
    if (!coop) return bail(fail(KL_ERR_UNSUPPORTED, "device lacks cooperative launch"));

    const int d = c.head_dim, g = c.n_heads / c.n_kv_heads;
    // (the per-sequence O projection gives every query head workgroups of its own)
    if (ncu < c.n_heads)
        return bail(fail(KL_ERR_UNSUPPORTED, "n_heads %d exceeds the %d compute units",
                         c.n_heads, ncu));
    // the packed layout's geometry for this grid (one persistent workgroup per CU)
    const Geometry Gm = layout_geometry(c, ncu);
    S->nwg = ncu;
    S->Hp = Gm.Hp; S->Ap = Gm.Ap; S->Fp = Gm.Fp;
    const int KTH = Gm.KTH, KTO = g * Gm.KTq;
    S->Sg = Gm.Sg; S->Sc = Gm.Sc; S->Rc = Gm.Rc; S->KTc = Gm.KTc;
    S->qkv_rg = Gm.qkv_rg; S->o_rg = Gm.o_rg; S->gu_rg = Gm.gu_rg; S->down_rg = Gm.down_rg;
    S->head_rg = Gm.head_rg;
    S->off_attn_norm = Gm.off_attn_norm; S->off_ffn_norm = Gm.off_ffn_norm;
    S->off_qkv_bias = Gm.off_qkv_bias;
    S->off_qkv = Gm.off_qkv; S->off_o = Gm.off_o; S->off_gu = Gm.off_gu;
    S->off_down = Gm.off_down; S->layer_stride = Gm.layer_stride;
    S->off_router = Gm.off_router; S->gu_estride = Gm.gu_estride;
    S->down_estride = Gm.down_estride;
    S->off_final_norm = Gm.off_final_norm; S->off_lm_head = Gm.off_lm_head;
    S->off_embed = Gm.off_embed; S->off_dummy = Gm.off_dummy;
    S->arena_bytes = Gm.arena_bytes;
    TRY(hipMalloc(&S->arena, S->arena_bytes));

    // grid: one persistent workgroup per CU
    lds_layout_for(*S);
    if (S->lds_bytes > 160 * 1024 - 256)
        return bail(fail(KL_ERR_UNSUPPORTED, "LDS need %d bytes exceeds 160 KiB", S->lds_bytes));
    int per_cu = 0;
    TRY(step_kernel_setup(c.head_dim, c.n_heads / c.n_kv_heads, S->lds_bytes, &per_cu));
    if (per_cu < 1) return bail(fail(KL_ERR_UNSUPPORTED, "step kernel does not fit on a CU"));

    // K slices of the batched products (they depend on the grid, not on the batch)
    const int nkv = c.n_kv_heads;
    const int qkv_rows = nkv * S->qkv_rg * kTileRows;
    S->KSo = batched_k_slices(nkv, KTO, S->o_rg / 2, S->nwg);
    S->KSd = batched_k_slices(S->Sc, S->KTc, S->down_rg / 2, S->nwg);
    S->KSg = folded_k_slices(KTH, 1, S->gu_rg / 2, S->nwg);
    S->KSq = folded_k_slices(KTH, 1, qkv_rows / 16, S->nwg);

    // step scratch for the largest batch, zeroed; the device error word
    S->scratch_bytes = plan_scratch(*S, c.max_batch).total;
    TRY(hipMalloc(&S->scratch, S->scratch_bytes));
    TRY(hipMemsetAsync(S->scratch, 0, S->scratch_bytes, s));
    TRY(hipMalloc(&S->err, 256));
    TRY(hipMemsetAsync(S->err, 0, 256, s));
    S->epoch = reinterpret_cast<unsigned *>(reinterpret_cast<uint8_t *>(S->err) + 128);
    TRY(hipMalloc(&S->keys, (size_t)2 * c.max_batch * sizeof(unsigned long long)));
    TRY(hipMemsetAsync(S->keys, 0, (size_t)2 * c.max_batch * sizeof(unsigned long long), s));
    {
        const unsigned first_tag = 1;
        TRY(hipMemcpyAsync(S->epoch, &first_tag, sizeof first_tag, hipMemcpyHostToDevice, s));
        TRY(hipStreamSynchronize(s));
    }
    // this device's copy of the library's static scratch (the entry point
    // that allocates nothing), resolved once per device
    TRY(static_scratch_address(S->device, &S->static_scratch));

    // RoPE table (cos, sin) of pos * theta^(-2i/d), computed in double
    {
        const int half = d / 2;
        std::vector<float2> tab((size_t)c.max_seq * half);
        for (int p = 0; p < c.max_seq; ++p)
            for (int i = 0; i < half; ++i) {
                const double w = std::pow((double)c.rope_theta, -2.0 * i / (double)d);
                const double phi = (double)p * w;
                tab[(size_t)p * half + i] = make_float2((float)std::cos(phi), (float)std::sin(phi));
            }
        TRY(hipMalloc(&S->rope, tab.size() * sizeof(float2)));
        TRY(hipMemcpyAsync(S->rope, tab.data(), tab.size() * sizeof(float2),
                           hipMemcpyHostToDevice, s));
        TRY(hipStreamSynchronize(s));
    }

    // the arena starts zeroed: weights not set yet read as zero
    TRY(hipMemsetAsync(S->arena, 0, S->arena_bytes, s));

    // row maps (the same for every layer), kept on the device for set_layer
    {
        std::vector<int32_t> all;
        size_t at[5];
        for (int m = 0; m < 5; ++m) {
            const std::vector<int32_t> v = row_map(c, (RowMap)m);
            at[m] = all.size();
            all.insert(all.end(), v.begin(), v.end());
        }
        TRY(hipMalloc(&S->rowmaps, all.size() * sizeof(int32_t)));
        TRY(hipMemcpy(S->rowmaps, all.data(), all.size() * sizeof(int32_t),
                      hipMemcpyHostToDevice));
        for (int m = 0; m < 5; ++m) S->maps[m] = S->rowmaps + at[m];
    }
    TRY(hipDeviceSynchronize());
#undef TRY
    *out = S;
    return KL_OK;
}

kl_status kl_model_set_layer(kl_state *S, int32_t l, const kl_layer_ptrs *w, void *stream) {
    g_last_error.clear();
    if (!S || !w) return fail(KL_ERR_INVALID_ARGUMENT, "state and weights must not be NULL");
    const kl_config &c = S->cfg;
    if (l < 0 || l >= c.n_layers)
        return fail(KL_ERR_INVALID_ARGUMENT, "layer %d outside [0, %d)", l, c.n_layers);
    kl_status st = check_layer_ptrs(*w, l, c.qkv_bias != 0, c.n_experts > 1);
    if (st != KL_OK) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const kl_layer_ptrs &Lw = *w;
    uint8_t *Lb = S->arena + (size_t)l * S->layer_stride;
    const auto u16 = [](const void *p) { return reinterpret_cast<const uint16_t *>(p); };
    hipError_t pe = launch_gain_to_f32(reinterpret_cast<float *>(Lb + S->off_attn_norm),
                                       u16(Lw.attn_norm), c.hidden, S->Hp, s);
    if (pe == hipSuccess)
        pe = launch_gain_to_f32(reinterpret_cast<float *>(Lb + S->off_ffn_norm),
                                u16(Lw.ffn_norm), c.hidden, S->Hp, s);
    if (pe == hipSuccess && c.qkv_bias)
        pe = launch_pack_bias(reinterpret_cast<float *>(Lb + S->off_qkv_bias),
                              c.n_kv_heads * S->qkv_rg * kTileRows, S->maps[kMapQkv], u16(Lw.bq),
                              u16(Lw.bk), u16(Lw.bv), s);
    // the packed matrices of the layer (kl_layout.h: layer_pack_jobs)
    const uint16_t *srcs[] = {u16(Lw.wq),     u16(Lw.wk),   u16(Lw.wv),     u16(Lw.wo),
                              u16(Lw.w_gate), u16(Lw.w_up), u16(Lw.w_down), nullptr,
                              u16(Lw.w_router)};
    for (const PackJob &J : layer_pack_jobs(c, layout_geometry(c, S->nwg))) {
        if (pe != hipSuccess) break;
        const uint16_t *p[3];
        for (int k = 0; k < 3; ++k) p[k] = J.src[k] == kSrcNone ? nullptr : srcs[J.src[k]] + J.col0;
        pe = launch_pack_rows(reinterpret_cast<uint16_t *>(Lb + J.dst), J.n_rg, J.KT, J.K, J.ld,
                              S->maps[J.map], p[0], p[1], p[2], s);
    }
    if (pe != hipSuccess)
        return fail(KL_ERR_HIP, "packing layer %d failed: %s", l, hipGetErrorString(pe));
    HIP_TRY(hipStreamSynchronize(s));
    return KL_OK;
}

kl_status kl_model_set_globals(kl_state *S, const void *embed, const void *final_norm,
                               const void *lm_head, void *stream) {
    g_last_error.clear();
    if (!S || !embed || !final_norm || !lm_head)
        return fail(KL_ERR_INVALID_ARGUMENT, "state and weight pointers must not be NULL");
    if (!aligned(embed, 2) || !aligned(final_norm, 2) || !aligned(lm_head, 2))
        return fail(KL_ERR_INVALID_ARGUMENT, "weight pointers must be 2-byte aligned");
    const kl_config &c = S->cfg;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t pe = launch_gain_to_f32(reinterpret_cast<float *>(S->arena + S->off_final_norm),
                                       reinterpret_cast<const uint16_t *>(final_norm), c.hidden,
                                       S->Hp, s);
    if (pe == hipSuccess) {
        const PackJob J = head_pack_job(c, layout_geometry(c, S->nwg));
        pe = launch_pack_rows(reinterpret_cast<uint16_t *>(S->arena + J.dst), J.n_rg, J.KT, J.K,
                              J.ld, S->maps[J.map],
                              reinterpret_cast<const uint16_t *>(lm_head) + J.col0, nullptr,
                              nullptr, s);
    }
    if (pe == hipSuccess)
        pe = hipMemcpyAsync(S->arena + S->off_embed, embed, (size_t)c.vocab * c.hidden * 2,
                            hipMemcpyDeviceToDevice, s);
    if (pe != hipSuccess)
        return fail(KL_ERR_HIP, "packing the globals failed: %s", hipGetErrorString(pe));
    HIP_TRY(hipStreamSynchronize(s));
    return KL_OK;
}

kl_status kl_load_model(const kl_config *cfg, const kl_weight_ptrs *w, void *stream,
                        kl_state **out) {
    g_last_error.clear();
    if (!out) return fail(KL_ERR_INVALID_ARGUMENT, "out is NULL");
    *out = nullptr;
    kl_status st = validate_config(cfg);
    if (st != KL_OK) return st;
    if (!w || !w->embed || !w->final_norm || !w->lm_head || !w->layers)
        return fail(KL_ERR_INVALID_ARGUMENT, "weight pointers must not be NULL");
    if (!aligned(w->embed, 2) || !aligned(w->final_norm, 2) || !aligned(w->lm_head, 2))
        return fail(KL_ERR_INVALID_ARGUMENT, "weight pointers must be 2-byte aligned");
    for (int l = 0; l < cfg->n_layers; ++l) {
        st = check_layer_ptrs(w->layers[l], l, cfg->qkv_bias != 0, cfg->n_experts > 1);
        if (st != KL_OK) return st;
    }
    kl_state *S = nullptr;
    st = kl_model_create(cfg, &S);
    if (st != KL_OK) return st;
    for (int l = 0; l < cfg->n_layers && st == KL_OK; ++l)
        st = kl_model_set_layer(S, l, &w->layers[l], stream);
    if (st == KL_OK) st = kl_model_set_globals(S, w->embed, w->final_norm, w->lm_head, stream);
    if (st != KL_OK) {
        const std::string msg = g_last_error;
        free_state(S);
        g_last_error = msg;
        return st;
    }
    *out = S;
    return KL_OK;
}

// Host-side checks shared by the step entry points (nothing is enqueued on
// failure).
static kl_status check_step_args(kl_state *st, const int32_t *token_ids,
                                 const int32_t *positions, int32_t batch, const kl_kv_cache *kv,
                                 const float *logits_out, const float *hidden_out, int32_t mode) {
    if (!st) return fail(KL_ERR_INVALID_ARGUMENT, "state is NULL");
    if (!token_ids || !positions || !logits_out || !kv || !kv->k || !kv->v)
        return fail(KL_ERR_INVALID_ARGUMENT, "token_ids, positions, kv, kv->k, kv->v and "
                                             "logits_out must not be NULL");
    if (!aligned(token_ids, 4) || !aligned(positions, 4) || !aligned(logits_out, 4) ||
        (hidden_out && !aligned(hidden_out, 4)))
        return fail(KL_ERR_INVALID_ARGUMENT, "int32/fp32 buffers must be 4-byte aligned");
    if (!aligned(kv->k, 16) || !aligned(kv->v, 16))
        return fail(KL_ERR_INVALID_ARGUMENT, "KV cache buffers must be 16-byte aligned");
    const kl_config &c = st->cfg;
    if (batch < 1 || batch > c.max_batch)
        return fail(KL_ERR_INVALID_ARGUMENT, "batch %d outside [1, max_batch=%d]", batch,
                    c.max_batch);
    if (kv->batch < batch)
        return fail(KL_ERR_INVALID_ARGUMENT, "kv batch extent %d < batch %d", kv->batch, batch);
    if (kv->capacity < 1 || kv->capacity > c.max_seq)
        return fail(KL_ERR_INVALID_ARGUMENT, "kv capacity %d outside [1, max_seq=%d]",
                    kv->capacity, c.max_seq);
    if (mode != KL_MODE_PER_LAYER && mode != KL_MODE_LOOPED && mode != KL_MODE_PER_OP &&
        mode != KL_MODE_PER_LAYER_GRAPH)
        return fail(KL_ERR_INVALID_ARGUMENT, "unknown mode %d", mode);
    // (a token's experts are chosen in the gate/up phase and kept in LDS
    // for the down phase of the same launch, on the per-sequence path)
    if (c.n_experts > 1 && (batch >= kMfmaBatch || mode == KL_MODE_PER_OP))
        return fail(KL_ERR_UNSUPPORTED, "a mixture of experts runs with batch < %d and not in "
                                        "the per-op schedule", kMfmaBatch);
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev != st->device)
        return fail(KL_ERR_INVALID_ARGUMENT, "current device %d is not the model's device %d",
                    dev, st->device);
    return KL_OK;
}

// The step's parameters with its scratch in 'base' (laid out by 'plan').
static StepParams step_params(const kl_state &st, uint8_t *base, const ScratchPlan &plan,
                              const int32_t *token_ids, const int32_t *positions, int32_t batch,
                              const kl_kv_cache *kv, float *logits_out, float *hidden_out) {
    StepParams P = base_params(st);
    bind_scratch(P, base, plan, st);
    P.tokens = token_ids; P.positions = positions; P.B = batch;
    P.kc = reinterpret_cast<uint16_t *>(kv->k); P.vc = reinterpret_cast<uint16_t *>(kv->v);
    P.kv_batch = kv->batch; P.cap = kv->capacity;
    P.logits = logits_out; P.hidden_out = hidden_out;
    P.C = std::max(1, st.Sg / batch);
    P.batched = batch >= st.batched_from ? 1 : 0;
    // (several sequences share a GEMV pass; the partial sums' place differs
    // between the two paths)
    P.multi = !P.batched && batch >= 2 && batch <= kMultiSeq && st.multi_ok ? 1 : 0;
    P.lds_red = P.batched ? st.lds_red : st.lds_red_seq;
    return P;
}

// The launches of one step in schedule 'mode'.
static hipError_t launch_schedule(const StepParams &P, int32_t mode, int lds, hipStream_t s) {
    const int L = P.L;
    const bool bat = P.batched != 0;
    hipError_t e = hipSuccess;
    if (mode == KL_MODE_LOOPED)
        return launch_step(P, 0, L, kPhEmbed | kPhLayer | kPhHead, true, lds, s);
    e = launch_step(P, 0, 0, kPhEmbed, false, lds, s);
    if (mode == KL_MODE_PER_LAYER) {
        for (int l = 0; l < L && e == hipSuccess; ++l)
            e = launch_step(P, l, l + 1, kPhLayer, launch_waits_inside(kPhLayer, bat, P.C), lds, s);
    } else {
        const int ops[] = {kPhQkv, kPhAttn, kPhOproj, kPhGateUp, kPhDown};
        for (int l = 0; l < L && e == hipSuccess; ++l)
            for (int ph : ops)
                if (e == hipSuccess)
                    e = launch_step(P, l, l + 1, ph, launch_waits_inside(ph, bat, P.C), lds, s);
    }
    if (e == hipSuccess)
        e = launch_step(P, 0, 0, kPhHead, launch_waits_inside(kPhHead, bat, P.C), lds, s);
    return e;
}

// KL_MODE_PER_LAYER_GRAPH: the per-layer schedule's L + 2 launches as one
// graph (kernel nodes in a chain; the nodes whose workgroups wait on each
// other cooperative), built for the caller's buffers on first use and
// replayed while they stay the same.  Every step of a model computes with the
// same arguments apart from those buffers: the tags of the hand-offs are read
// from device memory.
static kl_status launch_layer_graph(kl_state *st, const StepParams &P, hipStream_t s) {
    const void *key[10] = {P.tokens, P.positions, (const void *)(intptr_t)P.B, P.kc, P.vc,
                           (const void *)(intptr_t)P.kv_batch, (const void *)(intptr_t)P.cap,
                           P.logits, P.hidden_out, P.trace};
    bool same = st->graph_exec != nullptr;
    for (int i = 0; i < 10 && same; ++i) same = st->graph_key[i] == key[i];
    if (!same) {
        if (st->graph_exec) HIP_TRY(hipGraphExecDestroy(st->graph_exec));
        if (st->graph) HIP_TRY(hipGraphDestroy(st->graph));
        st->graph_exec = nullptr;
        st->graph = nullptr;
        HIP_TRY(hipGraphCreate(&st->graph, 0));
        const bool bat = P.batched != 0;
        const int lds = st->lds_bytes;
        hipGraphNode_t prev = nullptr, node = nullptr;
        HIP_TRY(add_step_node(st->graph, &node, nullptr, P, 0, 0, kPhEmbed, false, lds));
        for (int l = 0; l < P.L; ++l) {
            prev = node;
            HIP_TRY(add_step_node(st->graph, &node, &prev, P, l, l + 1, kPhLayer,
                                  launch_waits_inside(kPhLayer, bat, P.C), lds));
        }
        prev = node;
        HIP_TRY(add_step_node(st->graph, &node, &prev, P, 0, 0, kPhHead,
                              launch_waits_inside(kPhHead, bat, P.C), lds));
        HIP_TRY(hipGraphInstantiate(&st->graph_exec, st->graph, nullptr, nullptr, 0));
        for (int i = 0; i < 10; ++i) st->graph_key[i] = key[i];
    }
    HIP_TRY(hipGraphLaunch(st->graph_exec, s));
    return KL_OK;
}

// One decode step: validation, the scratch binding, the launches of 'mode'.
// With no_alloc the step's scratch is the library's static scratch of this
// device (cleared first by a fill kernel on the stream), else the state's.
static kl_status enqueue_step(kl_state *st, const int32_t *token_ids, const int32_t *positions,
                              int32_t batch, const kl_kv_cache *kv, float *logits_out,
                              float *hidden_out, void *stream, int32_t mode, bool no_alloc) {
    g_last_error.clear();
    kl_status stt = check_step_args(st, token_ids, positions, batch, kv, logits_out, hidden_out,
                                    mode);
    if (stt != KL_OK) return stt;
    const kl_config &c = st->cfg;
    ScratchPlan plan;
    uint8_t *base;
    if (no_alloc) {
        plan = plan_scratch(*st, batch);
        if (plan.total > kStaticScratchBytes)
            return fail(KL_ERR_UNSUPPORTED,
                        "this step needs %zu bytes of scratch; the static scratch holds %zu "
                        "(use kl_decode_step)", plan.total, kStaticScratchBytes);
        if (!st->static_scratch)
            return fail(KL_ERR_HIP, "the static scratch of device %d is not resolved", st->device);
        base = st->static_scratch;
    } else {
        plan = plan_scratch(*st, c.max_batch);
        base = st->scratch;
    }
    const StepParams P = step_params(*st, base, plan, token_ids, positions, batch, kv, logits_out,
                                     hidden_out);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    // (the static scratch holds whatever the last call on this device left:
    // it starts from zero like a fresh allocation)
    if (mode == KL_MODE_PER_LAYER_GRAPH) {
        if (no_alloc)
            return fail(KL_ERR_INVALID_ARGUMENT, "the graph schedule is not available without "
                                                 "allocation (building a graph allocates)");
        return launch_layer_graph(st, P, s);
    }
    if (no_alloc) HIP_TRY(launch_zero(base, plan.total, s));
    HIP_TRY(launch_schedule(P, mode, st->lds_bytes, s));
    return KL_OK;
}

kl_status kl_decode_step(kl_state *st, const int32_t *token_ids, const int32_t *positions,
                         int32_t batch, const kl_kv_cache *kv, float *logits_out,
                         float *hidden_out, void *stream, int32_t mode) {
    return enqueue_step(st, token_ids, positions, batch, kv, logits_out, hidden_out, stream, mode,
                        false);
}

kl_status kl_decode_step_noalloc(kl_state *st, const int32_t *token_ids,
                                 const int32_t *positions, int32_t batch, const kl_kv_cache *kv,
                                 float *logits_out, float *hidden_out, void *stream,
                                 int32_t mode) {
    return enqueue_step(st, token_ids, positions, batch, kv, logits_out, hidden_out, stream, mode,
                        true);
}

kl_status kl_decode_greedy(kl_state *st, const int32_t *token_ids, const int32_t *positions,
                           int32_t batch, int32_t n_steps, const kl_kv_cache *kv,
                           int32_t *tokens_out, float *logits_out, void *stream, int32_t mode) {
    g_last_error.clear();
    kl_status stt = check_step_args(st, token_ids, positions, batch, kv, logits_out, nullptr, mode);
    if (stt != KL_OK) return stt;
    if (n_steps < 1) return fail(KL_ERR_INVALID_ARGUMENT, "n_steps %d < 1", n_steps);
    if (mode == KL_MODE_PER_LAYER_GRAPH)
        return fail(KL_ERR_INVALID_ARGUMENT, "the token loop runs the looped, per-layer or "
                                             "per-op schedule");
    if (!tokens_out || !aligned(tokens_out, 4))
        return fail(KL_ERR_INVALID_ARGUMENT, "tokens_out must be a 4-byte aligned pointer");
    const kl_config &c = st->cfg;
    StepParams P = step_params(*st, st->scratch, plan_scratch(*st, c.max_batch), token_ids,
                               positions, batch, kv, logits_out, nullptr);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    // step n: positions + n; its head leaves the argmax keys in keys[n % 2],
    // from which step n + 1's embedding takes its tokens (recording them as
    // tokens_out[n])
    for (int32_t n = 0; n < n_steps; ++n) {
        P.pos_add = n;
        P.amax = st->keys + (size_t)(n % 2) * c.max_batch;
        P.tok_keys = n == 0 ? nullptr : st->keys + (size_t)((n - 1) % 2) * c.max_batch;
        P.tok_emit = n == 0 ? nullptr : tokens_out + (size_t)(n - 1) * batch;
        HIP_TRY(launch_schedule(P, mode, st->lds_bytes, s));
    }
    HIP_TRY(launch_emit_tokens(tokens_out + (size_t)(n_steps - 1) * batch,
                               st->keys + (size_t)((n_steps - 1) % 2) * c.max_batch, batch, s));
    return KL_OK;
}

kl_status kl_get_device_error(kl_state *st, int32_t *code) {
    g_last_error.clear();
    if (!st || !code) return fail(KL_ERR_INVALID_ARGUMENT, "state and code must not be NULL");
    HIP_TRY(hipDeviceSynchronize());
    int32_t v = 0;
    HIP_TRY(hipMemcpy(&v, st->err, sizeof v, hipMemcpyDeviceToHost));
    *code = v;
    if (v == 0) return KL_OK;
    HIP_TRY(hipMemset(st->err, 0, sizeof(int32_t)));
    if (v & KL_DEVERR_BARRIER) {
        // a timed-out barrier leaves its counters mid-count: start them afresh
        // (the static scratch is cleared by every call that uses it)
        const ScratchPlan pl = plan_scratch(*st, st->cfg.max_batch);
        HIP_TRY(hipMemset(st->scratch + pl.off_bar, 0, pl.off_cnt_end - pl.off_bar));
    }
    return fail(KL_ERR_DEVICE_FAULT, "device error word 0x%x", v);
}

kl_status kl_set_trace(kl_state *st, uint64_t *dev_buffer, int32_t max_phases) {
    g_last_error.clear();
    if (!st) return fail(KL_ERR_INVALID_ARGUMENT, "state is NULL");
    if (dev_buffer && (max_phases < 1 || !aligned(dev_buffer, 8)))
        return fail(KL_ERR_INVALID_ARGUMENT, "trace buffer needs max_phases >= 1, 8-byte alignment");
    st->trace = reinterpret_cast<unsigned long long *>(dev_buffer);
    st->trace_max = dev_buffer ? max_phases : 0;
    return KL_OK;
}

kl_status kl_read_stream(const void *buf, size_t bytes, int32_t workgroups, uint32_t *dev_out,
                         void *stream) {
    if (buf == nullptr || dev_out == nullptr)
        return fail(KL_ERR_INVALID_ARGUMENT, "kl_read_stream: null pointer");
    if ((reinterpret_cast<uintptr_t>(buf) & 15) != 0 || bytes % 16 != 0)
        return fail(KL_ERR_INVALID_ARGUMENT,
                    "kl_read_stream: buffer and size must be multiples of 16 bytes");
    if (workgroups < 1 || workgroups > 65536)
        return fail(KL_ERR_INVALID_ARGUMENT, "kl_read_stream: workgroups %d outside [1, 65536]",
                    workgroups);
    if (bytes == 0) return KL_OK;
    const hipError_t e = launch_read_stream(buf, bytes, workgroups, dev_out,
                                            reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? KL_OK : fail(KL_ERR_HIP, "kl_read_stream: %s", hipGetErrorString(e));
}

kl_status kl_get_info(const kl_state *st, kl_info *info) {
    if (!st || !info) return fail(KL_ERR_INVALID_ARGUMENT, "state and info must not be NULL");
    info->n_workgroups = st->nwg;
    info->threads_per_group = kThreads;
    info->lds_bytes = st->lds_bytes;
    info->attn_chunks_b1 = std::max(1, st->Sg);
    info->mfma_min_batch = st->batched_from;
    info->arena_bytes = (int64_t)st->arena_bytes;
    info->scratch_bytes = (int64_t)st->scratch_bytes;
    info->noalloc_scratch_bytes = (int64_t)plan_scratch(*st, st->cfg.max_batch).total;
    info->noalloc_scratch_limit = (int64_t)kStaticScratchBytes;
    return KL_OK;
}

void kl_free_model(kl_state *st) {
    if (!st) return;
    (void)hipDeviceSynchronize();
    free_state(st);
}

}  // extern "C"
