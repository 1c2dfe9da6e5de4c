/*
 * kl — one decode step of a Llama-style decoder-only transformer on one
 * AMD MI355X (gfx950), with kernel looping (arXiv 2410.23668).
 *
 * The paper's token step is Embedding -> L x Decoder -> Classifier (Sec. 2).
 * Each decoder layer is RMSNorm, the Q/K/V projections, RoPE, GQA attention
 * over the KV cache, the O projection with a residual add, RMSNorm, a SwiGLU
 * MLP and a second residual add.  The step runs in one of three schedules:
 *
 *   KL_MODE_PER_LAYER  one kernel launch per decoder layer (the layer-level
 *                      fusion baseline of Sec. 2, K0 called L times), plus one
 *                      launch for the embedding and one for the classifier:
 *                      L + 2 dispatches.
 *   KL_MODE_LOOPED     kernel looping (Sec. 2 and Sec. 3.2): the L chained
 *                      layer calls become one call of a kernel with an outer
 *                      loop over layers; the embedding and classifier run in
 *                      the same launch: 1 dispatch.  Kernel boundaries are
 *                      replaced by device-scope counters.
 *   KL_MODE_PER_OP     one launch per operator group of a layer (the many-
 *                      kernels-per-layer GPU schedule of Sec. 2, Fig. 3 (i)):
 *                      5 L + 2 dispatches.
 *   KL_MODE_PER_LAYER_GRAPH
 *                      the per-layer schedule's L + 2 launches recorded once as
 *                      a HIP graph and replayed (the graph alternative of the
 *                      related work, Sec. 5): rebuilt when the caller's
 *                      buffers (tokens, positions, batch, cache, outputs,
 *                      trace) differ from the last call's; one graph per
 *                      state.  Not available to kl_decode_step_noalloc or
 *                      kl_decode_greedy.
 *
 * All modes run the same device code with the same work partition, so for the
 * same inputs they produce bit-identical logits, hidden states and KV writes.
 *
 * Conventions.  All tensors are row-major.  "dev" pointers are device memory
 * of the current HIP device; "host" pointers are host memory.  bf16 values are
 * passed as their 16-bit patterns.  Streams are hipStream_t passed as void*
 * (NULL = the default stream).  Functions returning kl_status return KL_OK or
 * a negative code; on a negative code nothing was enqueued and kl_last_error()
 * describes the problem.  The library is built for gfx950 only.
 */
#ifndef KL_H
#define KL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KL_OK = 0,
    KL_ERR_INVALID_ARGUMENT = -1,  /* null / misaligned pointer, bad size, bad mode  */
    KL_ERR_UNSUPPORTED = -2,       /* a shape this build does not implement           */
    KL_ERR_OUT_OF_MEMORY = -3,     /* device allocation failed                        */
    KL_ERR_HIP = -4,               /* a HIP runtime call failed (message has details) */
    KL_ERR_DEVICE_FAULT = -5       /* reported by kl_get_device_error                 */
} kl_status;

typedef enum {
    KL_MODE_PER_LAYER = 0,
    KL_MODE_LOOPED = 1,
    KL_MODE_PER_OP = 2,
    KL_MODE_PER_LAYER_GRAPH = 3
} kl_mode;

/* Bits of the device error word (kl_get_device_error).  A sequence with a bad
 * token or position is skipped: none of its K/V slots is written and its
 * logits (and hidden state) are NaN; the other sequences of the step are
 * computed normally. */
#define KL_DEVERR_TOKEN    1   /* a token id outside [0, vocab)                              */
#define KL_DEVERR_POSITION 2   /* a position outside [0, capacity) or >= max_seq             */
#define KL_DEVERR_BARRIER  4   /* a grid barrier waited longer than its watchdog allows      */

/* Model shape.  Supported: head_dim 64 or 128, n_heads a multiple of
 * n_kv_heads with n_heads / n_kv_heads one of 1, 2, 4, 8 (and 3 with
 * head_dim 128), n_heads at most the GPU's compute units, every dimension
 * >= 1 and hidden, ffn_dim multiples of 8.  max_batch bounds the batch of a
 * step; max_seq bounds positions (the RoPE table covers [0, max_seq)).
 * qkv_bias: 1 if the Q/K/V projections carry biases (the Qwen2.5 variant of
 * Table 2), else 0.  Tied embeddings (Llama 3.2) need no flag: pass the
 * embedding table as the LM head.
 * n_experts, top_k: a mixture of experts in place of the SwiGLU MLP (the
 * Mixtral 8x7B variant of Table 2): 2..8 experts per layer, top_k 1 or 2
 * of them per token, chosen by a router and weighted by the softmax of the
 * chosen router logits (the lowest index first among equal logits); 0 (or
 * 1) experts: the dense MLP.  With experts, steps run with batch < 8 and not
 * in KL_MODE_PER_OP (KL_ERR_UNSUPPORTED otherwise). */
typedef struct {
    int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
    float rope_theta, rms_eps;
    int32_t max_batch, max_seq;
    int32_t qkv_bias;
    int32_t n_experts, top_k;
} kl_config;

/* One decoder layer's weights: dev bf16, nn.Linear layout [out][in].
 *   attn_norm, ffn_norm [hidden]
 *   wq [n_heads*head_dim][hidden], wk, wv [n_kv_heads*head_dim][hidden]
 *   wo [hidden][n_heads*head_dim]
 *   w_gate, w_up [ffn_dim][hidden], w_down [hidden][ffn_dim]
 *   bq [n_heads*head_dim], bk, bv [n_kv_heads*head_dim]: the Q/K/V biases,
 *   required with cfg.qkv_bias and ignored (may be NULL) without
 *   with n_experts > 1: w_gate, w_up [n_experts][ffn_dim][hidden],
 *   w_down [n_experts][hidden][ffn_dim] (the experts' MLPs, stacked) and
 *   w_router [n_experts][hidden]; w_router is ignored (may be NULL) without */
typedef struct {
    const void *attn_norm, *wq, *wk, *wv, *wo, *ffn_norm, *w_gate, *w_up, *w_down;
    const void *bq, *bk, *bv;
    const void *w_router;
} kl_layer_ptrs;

/* Whole model: dev bf16 embed [vocab][hidden], final_norm [hidden],
 * lm_head [vocab][hidden] (untied); layers is a host array of n_layers. */
typedef struct {
    const void *embed, *final_norm, *lm_head;
    const kl_layer_ptrs *layers;
} kl_weight_ptrs;

/* Caller-owned KV cache: dev bf16 k and v, each
 * [n_layers][batch][n_kv_heads][capacity][head_dim], holding post-RoPE keys.
 * 'batch' is the allocated batch extent (>= the step's batch), 'capacity'
 * the allocated positions per sequence.  16-byte aligned. */
typedef struct {
    void *k, *v;
    int32_t batch, capacity;
} kl_kv_cache;

typedef struct kl_state kl_state;

/* Read-only facts about a loaded model (for benches and tests). */
typedef struct {
    int32_t n_workgroups;       /* persistent grid size used by every mode        */
    int32_t threads_per_group;
    int32_t lds_bytes;          /* dynamic LDS per workgroup                       */
    int32_t attn_chunks_b1;     /* KV chunks per (sequence, KV head) at batch 1    */
    int32_t mfma_min_batch;     /* steps with batch >= this run the weight products
                                   on the matrix cores                             */
    int64_t arena_bytes;        /* packed weights + gains                          */
    int64_t scratch_bytes;      /* activations, partials, counters                 */
    int64_t noalloc_scratch_bytes;  /* scratch a kl_decode_step_noalloc call at
                                       max_batch needs                             */
    int64_t noalloc_scratch_limit;  /* bytes of the static scratch                  */
} kl_info;

/* Load a model: validates cfg, allocates the packed weight arena, the RoPE
 * table and the step scratch on the current device, and repacks the caller's
 * weights into the gfx950 layout with kernels on 'stream'.  Returns after the
 * stream has finished the packing, so the caller may free the source weights.
 * The grouped weights of all layers are laid out linearly in one arena (the
 * grouping rule of Sec. 3.2, Eq. 3, with the linear layout it suggests).
 * On success *out owns every allocation; release with kl_free_model. */
kl_status kl_load_model(const kl_config *cfg, const kl_weight_ptrs *weights, void *stream,
                        kl_state **out);

/* Incremental loading, for models whose source weights cannot sit in device
 * memory beside the packed copy (e.g. the 70B shape on one GPU): the same
 * result as kl_load_model, one layer at a time.
 *   kl_model_create      validates cfg and allocates everything kl_load_model
 *                        allocates; the weights start as zeros.
 *   kl_model_set_layer   packs layer 'layer' (0 <= layer < n_layers) from the
 *                        caller's device pointers (layout of kl_layer_ptrs);
 *                        returns after the packing finished on 'stream', so
 *                        the caller may free the source right away.
 *   kl_model_set_globals packs the embedding, final norm and LM head (layouts
 *                        of kl_weight_ptrs), likewise synchronously.
 * Steps may run once every layer and the globals are set (earlier steps
 * compute with zero weights).  Errors as for kl_load_model; a failed set call
 * leaves the model usable for another attempt. */
kl_status kl_model_create(const kl_config *cfg, kl_state **out);
kl_status kl_model_set_layer(kl_state *st, int32_t layer, const kl_layer_ptrs *weights,
                             void *stream);
kl_status kl_model_set_globals(kl_state *st, const void *embed, const void *final_norm,
                               const void *lm_head, void *stream);

/* Enqueue one decode step on 'stream' (asynchronous): the token step of the
 * paper's Sec. 2 and Fig. 3 (Embedding -> L x Decoder -> Classifier), for
 * every sequence of the batch.  In KL_MODE_LOOPED the L decoder-layer calls
 * are collapsed into one call of the looped kernel (Sec. 3.2: the grouped
 * per-layer arguments become one linearly laid-out argument, the call sites
 * collapse into one); the other modes issue one launch per layer or per
 * operator group.  Every mode computes the same bits.
 *   token_ids  dev int32 [batch]   token of each sequence
 *   positions  dev int32 [batch]   position p of the new token; the step writes
 *                                  K/V slot p of every layer and attends over
 *                                  slots 0..p
 *   batch      1 <= batch <= min(max_batch, kv->batch)
 *   kv         caller's cache (layout above); capacity <= max_seq
 *   logits_out dev fp32 [batch][vocab]
 *   hidden_out dev fp32 [batch][hidden] or NULL: the residual stream after the
 *              last layer (before the final norm)
 *   mode       a kl_mode
 * Host-checkable errors (NULL or misaligned pointers, batch or capacity out
 * of range, an unknown mode, the wrong current device) return a negative
 * status with nothing enqueued.  Out-of-range token ids or positions can only
 * be seen on the device: they set bits in the device error word, and that
 * sequence is skipped as described with the bits.  One step may be in flight
 * per state; the caller's buffers are borrowed until the step completes in
 * stream order. */
kl_status kl_decode_step(kl_state *st, const int32_t *token_ids, const int32_t *positions,
                         int32_t batch, const kl_kv_cache *kv, float *logits_out,
                         float *hidden_out, void *stream, int32_t mode);

/* Greedy token loop: n_steps decode steps in a row on 'stream', each one's
 * sampled tokens feeding the next on the device (the Sampling block, executed
 * once per output token, Sec. 2 and Fig. 3; the paper does not fix the
 * sampler: greedy, the largest logit, the lowest index on ties).  Step n runs
 * at positions[b] + n on the tokens step n - 1 sampled (step 0 on token_ids),
 * writes K/V slot positions[b] + n of every layer, and samples in the LM
 * head's epilogue (no separate kernel, no host round trip).
 *   token_ids, positions, batch, kv, mode   as for kl_decode_step
 *   n_steps     >= 1
 *   tokens_out  dev int32 [n_steps][batch]: the token sampled at each step
 *   logits_out  dev fp32 [batch][vocab]: every step's logits in turn (the last
 *               step's remain)
 * A sequence whose token or position is out of range at some step is skipped
 * from then on (error bits as for kl_decode_step; it samples token -1).  Same
 * host-side errors as kl_decode_step, plus n_steps < 1 or a NULL or
 * misaligned tokens_out; nothing is enqueued then. */
kl_status kl_decode_greedy(kl_state *st, const int32_t *token_ids, const int32_t *positions,
                           int32_t batch, int32_t n_steps, const kl_kv_cache *kv,
                           int32_t *tokens_out, float *logits_out, void *stream, int32_t mode);

/* kl_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same arguments, results and errors, bit-identical outputs, and it calls
 * no allocating routine.  Its step scratch is not the state's but a static
 * array of the library, one per device, of kl_info.noalloc_scratch_limit bytes
 * (32 MiB), held until the process ends; a step that needs more (see
 * kl_info.noalloc_scratch_bytes: e.g. the 70B shape on the matrix-core path) returns
 * KL_ERR_UNSUPPORTED with nothing enqueued.  Each call first clears the
 * scratch it uses with a fill kernel on 'stream' (one extra launch), so no
 * state carries over from an earlier call.  Every call on a device shares
 * that device's array: calls that may overlap in time on one device (other
 * streams, other threads, other states) race and must be serialized by the
 * caller. */
kl_status kl_decode_step_noalloc(kl_state *st, const int32_t *token_ids,
                                 const int32_t *positions, int32_t batch, const kl_kv_cache *kv,
                                 float *logits_out, float *hidden_out, void *stream,
                                 int32_t mode);

/* Bytes of ONE of the K or V buffers for the given batch and capacity
 * (0 if cfg is invalid). */
size_t kl_kv_cache_bytes(const kl_config *cfg, int32_t batch, int32_t capacity);

/* Synchronizes the device, returns the device error word in *code (KL_DEVERR_*
 * bits, 0 = none) and clears it.  Returns KL_ERR_DEVICE_FAULT when *code != 0. */
kl_status kl_get_device_error(kl_state *st, int32_t *code);

kl_status kl_get_info(const kl_state *st, kl_info *info);

/* Timeline of the phases, for profiling the schedules (the kind of
 * synchronization-cost breakdown of Sec. 2, Fig. 5).  While a buffer is set,
 * every later launch writes, for phase i < max_phases of the launch (in the
 * order embed, then qkv, attn, oproj, gateup, down per layer, then head) and
 * workgroup w, s_memrealtime stamps (100 MHz ticks) into
 *   dev_buffer[(i * n_workgroups + w) * 4 + {0: phase end (every wave of the
 *   workgroup done; its writes complete where the phase ends on a barrier,
 *   issued where it hands tagged words to the next phase), 1: start of the
 *   wait for its inputs, 2: end of that wait, 3: inputs staged (in LDS on the
 *   per-sequence path; matrix-core path: the workgroup's share of the
 *   grid-wide step before the product, RMSNorm or SwiGLU fold, done; an
 *   attention phase: its chunk result published)}]
 * (slots a workgroup does not reach keep their old contents; a launch
 * overwrites the previous launch's entries).  The buffer (dev, uint64,
 * max_phases * n_workgroups * 4 entries) stays owned by the caller; pass NULL
 * to stop tracing. */
kl_status kl_set_trace(kl_state *st, uint64_t *dev_buffer, int32_t max_phases);

/* Measurement helper (no model involved): reads every byte of the device
 * buffer buf (bytes, both 16-byte aligned) once with the step kernel's
 * 16-byte non-temporal loads, 16 in flight per lane, on a grid of workgroups
 * x 512 lanes (1..65536 workgroups), and writes nothing the caller relies on
 * (dev_out, one device uint32, is at most written with an unspecified value).
 * Timed by the caller, it gives the read-stream rate this load pattern
 * reaches: the practical ceiling of a kernel whose traffic is one pass over
 * its weights (the roofline of Sec. 4.4's bandwidth comparison is the
 * nominal peak).  Asynchronous on stream; invalid arguments return
 * KL_ERR_INVALID_ARGUMENT with nothing enqueued. */
kl_status kl_read_stream(const void *buf, size_t bytes, int32_t workgroups, uint32_t *dev_out,
                         void *stream);

/* Frees everything the state owns (synchronizes the device first). NULL is a no-op. */
void kl_free_model(kl_state *st);

/* Message describing the last failing call on this thread ("" if none). */
const char *kl_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* KL_H */
