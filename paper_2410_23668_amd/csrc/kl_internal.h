// Internal interface between the host runtime (kl_host.cpp) and the device
// code (kl_device.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include "kl_layout.h"
#include "kl_sync.h"
#include <stddef.h>
#include <stdint.h>

namespace kl {

// Work geometry shared by host and device.
constexpr int kWaves = 8;                 // compute waves per workgroup
constexpr int kCtlWave = kWaves;          // the control wave: barriers and counters only
constexpr int kThreads = (kWaves + 1) * 64;   // threads per workgroup
constexpr int kOEarly = 4;               // O projection: waves that gather the merge (the rest load early)
constexpr int kRgBatch = 16;              // row groups reduced per LDS round
constexpr int kAttnLoads = 5;             // K (and V) loads per lane per sub-chunk, short attention chunks
constexpr int kAttnRing = 4;              // K (and V) slabs in flight per wave, streaming attention
constexpr int kCombBatch = 32;            // chunk partials loaded together when merging
// Batched steps (the matrix-core path) run the weight products on the matrix
// cores.  An activation x enters them as two bf16 terms, hi = bf16(x) and
// lo = bf16(x - hi), both multiplied into the same fp32 accumulators (about
// 16 significant bits of x instead of 8).  Activations are staged in LDS in
// chunks of kGemmChunkK columns for up to kGemmBatch sequences at a time,
// weight rows in blocks of 16.
constexpr int kMfmaBatch = 8;
// Up to kMultiSeq sequences share one pass of the GEMV engine: each weight
// tile is applied to every staged vector, so the weights stream once (8B
// shape, 4096 cached positions: 3.06, 3.52, 3.91, 4.35 ms at batch 1-4,
// against 5.0 ms on the matrix-core path).  Dense models take the
// matrix-core path from batch kMultiSeq + 1 on, or from kBatchedFrom where
// the LDS cannot hold the shared pass's vectors beside the matrix-core
// engine's area (one sequence per pass: 5.61 ms at batch 2).  A mixture of
// experts keeps the GEMV path below kMfmaBatch (its experts are chosen per
// token on that path).
constexpr int kMultiSeq = 4;
constexpr int kBatchedFrom = 2;
constexpr int kGemmBatch = 32;
constexpr int kGemmChunkK = 512;
constexpr int kActStride = kGemmChunkK + 8;   // bf16 per staged activation row (bank spread)
constexpr int kGemmMaxBlk = 4;            // 16-row blocks per wave per pass over the weights
constexpr int kMaxKSlices = 16;           // K slices of a batched product (partial sums)
constexpr int kGemmResidentK = 2 * kGemmChunkK;   // K columns a workgroup keeps resident
// LDS of the batched path (bytes): two activation chunks of both terms, and
// per-wave weight re-layout slots (2 KiB)
constexpr int kGemmActBytes = kGemmBatch * kActStride * 2;   // one term of one chunk
constexpr int kGemmLdsBytes = 4 * kGemmActBytes + kWaves * 2048;
constexpr int kNormCntStride = 64;        // words between batched RMSNorm slice counters
constexpr int kMaxGroup = 8;              // max query heads per KV head
constexpr int kMergeChunks = 32;          // attention chunk results merged per LDS round
constexpr int kDownGather = 8;            // tagged words per control-wave lane per gather round
constexpr int kBarGroups = kSyncBarGroups;   // first level of the grid barrier
constexpr int kBarBytes = 8192;           // barrier counters: kBarGroups lines of 256 B

// Phase selection bits of one launch of the step kernel.
enum : int {
    kPhEmbed = 1, kPhQkv = 2, kPhAttn = 4, kPhOproj = 8, kPhGateUp = 16, kPhDown = 32,
    kPhHead = 64,
    kPhLayer = kPhQkv | kPhAttn | kPhOproj | kPhGateUp | kPhDown,
};

// Everything one step needs, passed by value as the kernel argument.
struct StepParams {
    // shape
    int L, H, nq, nkv, d, F, V, group;
    int Hp, Ap, Fp;            // K extents padded to kTileK: hidden, n_heads*d, ffn
    int qkv_rg;                // row groups of one KV head's q/k/v block
    int o_rg;                  // row groups of one KV head's O-projection block (H / 8)
    int gu_rg;                 // row groups of the gate/up matrix (2 F / 8)
    int down_rg;               // row groups of one FFN column block of the down matrix
    int head_rg;               // row groups of the LM head
    float eps;
    int max_seq;
    // work partition (depends only on nwg and the shape)
    int Sg;                    // workgroups per KV head: w / Sg is the head
    int Sc, Rc, KTc;           // FFN column blocks, workgroups per block, k-tiles per block
    // packed weights
    const uint8_t *arena;      // layer 0 base
    size_t layer_stride;       // bytes between consecutive layers
    size_t off_attn_norm, off_ffn_norm, off_qkv, off_o, off_gu, off_down;
    size_t off_qkv_bias;       // fp32 Q/K/V biases in packed row order (qkv_bias models)
    int qkv_bias;
    // mixture of experts (E > 1): E experts per layer, topk per token; the
    // router (one packed row group) and expert e's gate/up and down matrices
    // at off_gu + e gu_estride, off_down + e down_estride
    int E, topk;
    size_t off_router, gu_estride, down_estride;
    const uint16_t *embed;     // [V][H] bf16, row-major
    const float *final_norm;   // [Hp]
    const uint16_t *lm_head;   // packed tiles
    const float2 *rope;        // [max_seq][d/2] (cos, sin)
    // step arguments
    const int32_t *tokens, *positions;
    // token loop (greedy sampling, one step per launch sequence):
    int pos_add;               // added to every position (step s of a loop: s)
    const unsigned long long *tok_keys;   // non-null: token b is the previous step's argmax
    int32_t *tok_emit;         // non-null: the embedding phase records the tokens it takes
    unsigned long long *amax;  // non-null: the head leaves each sequence's argmax key here
    int B;
    uint16_t *kc, *vc;         // [L][kv_batch][nkv][cap][d]
    int kv_batch, cap;
    float *logits, *hidden_out;
    // scratch
    long long *xf;             // [max_batch][Hp] residual stream, fixed point (2^-32 units)
    long long *xf2;            // batched path: the other residual buffer (the folds alternate)
    float *xpart;              // batched path: K-slice partials [ks][max_batch][Hp] (O, down)
    int xpart_stride;          // floats between consecutive K-slice partials
    int KSo, KSd;              // K slices of the batched O and down projections
    float *gpart;              // batched path: K-slice partials of the gate/up product
                               // [ks][max_batch][2F rows] and, at other times, of the
                               // q/k/v product [ks][max_batch][nkv * qkv_rg * 8 rows]
    int gpart_stride;          // floats between consecutive gate/up K-slice partials
    int qpart_stride;          // floats between consecutive q/k/v K-slice partials
    int KSg, KSq;              // K slices of the batched gate/up and q/k/v products
    float *ssp;                // batched path: sums of squares of the last RMSNorm step's
                               // rows per kGemmChunkK columns [max_batch][ceil(Hp / chunk)]
    float *q;                  // batched path: [B][nq*d] rotated queries
    float *part_o;             // batched path: attention chunk outputs [B*nkv*C][group*d]
    float *part_s;             // batched path: attention chunk (max, sum) [B*nkv*C][group][2]
    // per-sequence path (batch below the model's matrix-core batch): values handed between
    // workgroups as tagged words (value in the low 32 bits, the tag of the
    // writing step and layer in the high 32 bits)
    unsigned *epoch_ptr;       // device word: the current step's first tag (layer l's tag
                               // is *epoch_ptr + l; the step's last phase advances it)
    unsigned long long *q_ll;  // [B][nq*d] rotated queries (fp32)
    unsigned long long *kv_ll; // [B][nkv][d]: new key (d/2 words: bf16 dims i, i + d/2),
                               // then new value (d/2 words: bf16 dims 2j, 2j + 1)
    unsigned long long *po_ll; // [B][nkv][group][C][d + 2]: chunk outputs, then max and sum
    unsigned long long *m_ll;  // [B][Fp] SwiGLU output (fp32)
    // batched path: activations as bf16 hi and lo terms (hi + lo ~ the fp32 value)
    uint16_t *act, *act_lo;    // [max_batch][Hp] normalised activations
    uint16_t *actm, *actm_lo;  // [max_batch][Fp] SwiGLU output
    uint16_t *acto, *acto_lo;  // [max_batch][nq*d] attention output, when C == 1
    unsigned long long *bar;   // grid barrier counters (monotonic): group g at [32 (g + 1)]
    unsigned *cnt;             // local counters: [nkv] qkv, [nkv] attention, [Sc] gate/up,
                               // then the batched RMSNorm slices (256 bytes apart)
    int *err;                  // device error word
    const uint8_t *dummy;      // 16 readable bytes: target of the GEMV ring's spare loads
    int nwg;                   // grid size
    int lds_red, lds_sm, lds_bar;   // dynamic LDS layout (float offsets)
    int batched;               // this step runs the matrix-core path (set by the host)
    int multi;                 // per-sequence path: the B <= kMultiSeq sequences share each
                               // GEMV pass (set by the host)
    int C;                     // attention chunks per (sequence, KV head)
    unsigned long long *trace; // optional phase timestamps (see kl_set_trace), or null
    int trace_max;             // phases recorded per launch
};

typedef void (*StepKernel)(StepParams, int, int, int);
StepKernel step_kernel_d64(int group);
StepKernel step_kernel_d64_batched(int group);
StepKernel step_kernel_d128(int group);
StepKernel step_kernel_d128_batched(int group);

hipError_t launch_step(const StepParams &p, int first_layer, int last_layer, int phases,
                       bool cooperative, int lds_bytes, hipStream_t stream);
// Adds the same launch as a kernel node of graph g after 'dep' (null: none);
// cooperative nodes carry the graph's cooperative attribute.
hipError_t add_step_node(hipGraph_t g, hipGraphNode_t *node, const hipGraphNode_t *dep,
                         const StepParams &p, int first_layer, int last_layer, int phases,
                         bool cooperative, int lds_bytes);
hipError_t step_kernel_setup(int d, int group, int lds_bytes, int *max_blocks_per_cu);

// The static scratch of kl_decode_step_noalloc: one array per device, of
// this many bytes, held until the process ends.
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
// This device's address of the static scratch ('device' must be current);
// resolved with hipGetSymbolAddress once per device, then cached.
hipError_t static_scratch_address(int device, uint8_t **out);
// Zero 'bytes' (a multiple of 16, 16-byte aligned) at p with a fill kernel.
hipError_t launch_zero(void *p, size_t bytes, hipStream_t stream);
hipError_t launch_read_stream(const void *p, size_t bytes, int workgroups, uint32_t *out,
                              hipStream_t stream);

// tokens[b] = the token of argmax key keys[b] (-1 where there is none), b < n.
hipError_t launch_emit_tokens(int32_t *tokens, const unsigned long long *keys, int n,
                              hipStream_t stream);

hipError_t launch_pack_rows(uint16_t *dst, int n_rg, int kt, int K, int ld, const int32_t *rowmap,
                            const uint16_t *src0, const uint16_t *src1, const uint16_t *src2,
                            hipStream_t stream);
// dst[r] = fp32 bias of packed q/k/v row r (rowmap as for the matrix; the
// sources bq, bk, bv are source ids 0, 1, 2).
hipError_t launch_pack_bias(float *dst, int rows, const int32_t *rowmap, const uint16_t *bq,
                            const uint16_t *bk, const uint16_t *bv, hipStream_t stream);
hipError_t launch_gain_to_f32(float *dst, const uint16_t *src, int n, int npad,
                              hipStream_t stream);

}  // namespace kl
