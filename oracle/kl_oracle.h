/*
 * Oracle: the plain CPU definition of one decode step of a Llama-style
 * decoder-only transformer (the computation that kernel looping speeds up,
 * arXiv 2410.23668 Sec. 2: Embedding -> L x Decoder -> Classifier).
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests, the smoke check and the bench's CPU
 * baseline use it.  It shares no code with the HIP library.  Arithmetic is
 * fp64; weights and the KV cache are bf16 bit patterns (uint16), as in the
 * paper's BF16 workloads (Table 1).
 */
#ifndef KL_ORACLE_H
#define KL_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
    double rope_theta, rms_eps;
    /* mixture of experts (the Mixtral 8x7B entry of Table 2): n_experts > 1
     * experts per layer, top_k of them per token; 0 or 1: the dense MLP */
    int32_t n_experts, top_k;
} klo_config;

typedef struct {   /* bf16, nn.Linear layout [out][in], row-major */
    const uint16_t *attn_norm, *wq, *wk, *wv, *wo, *ffn_norm, *w_gate, *w_up, *w_down;
    /* optional Q/K/V biases (NULL: none), [n_heads*head_dim], [n_kv_heads*head_dim] x 2:
     * the Qwen2.5 variant of the decoder (its Table 2 entry) adds them to the projections */
    const uint16_t *bq, *bk, *bv;
    /* mixture of experts: the router [n_experts][hidden]; w_gate, w_up are then
     * n_experts stacked [ffn_dim][hidden] matrices and w_down n_experts
     * stacked [hidden][ffn_dim] */
    const uint16_t *w_router;
} klo_layer;

double   klo_bf16_to_f64(uint16_t h);
uint16_t klo_f64_to_bf16(double v);
void klo_bf16_to_f64_array(const uint16_t *src, double *dst, int64_t n);
void klo_f64_to_bf16_array(const double *src, uint16_t *dst, int64_t n);

void klo_rmsnorm(int32_t n, const double *x, const uint16_t *gain, double eps, double *u);
void klo_gemv(int32_t rows, int32_t cols, const uint16_t *w, const double *u, double *y,
              int32_t nthreads);
void klo_rope(int32_t head_dim, double theta, int32_t pos, double *y);
void klo_softmax(int32_t n, const double *s, double *a);
void klo_attention(int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, int32_t pos,
                   int32_t capacity, const double *q, const uint16_t *k_seq,
                   const uint16_t *v_seq, double *o);
void klo_swiglu(int32_t n, const double *gate, const double *up, double *m);
/* The experts a token is routed to: the top_k largest of the n router
 * logits (the lowest index first among equal ones), and their weights, the
 * softmax of their logits.  idx, w: [top_k]. */
void klo_route(int32_t n, int32_t top_k, const double *logits, int32_t *idx, double *w);

/* One decode step for batch sequences.  kcache/vcache: [L][kv_batch][n_kv][capacity][d]
 * bf16, updated at slot positions[b] of every layer.  logits: [batch][vocab],
 * hidden (nullable): [batch][hidden] (the residual stream before the final norm),
 * router (nullable, mixture of experts): [batch][L][n_experts] router logits.
 * Returns 0, or -1 when a token or position is out of range (nothing written). */
int32_t klo_decode_step(const klo_config *cfg, const uint16_t *embed,
                        const uint16_t *final_norm, const uint16_t *lm_head,
                        const klo_layer *layers, int32_t batch, const int32_t *tokens,
                        const int32_t *positions, uint16_t *kcache, uint16_t *vcache,
                        int32_t kv_batch, int32_t capacity, double *logits, double *hidden,
                        double *router, int32_t nthreads);

#ifdef __cplusplus
}
#endif
#endif
