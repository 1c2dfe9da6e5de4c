/*
 * Oracle for one decode step of a Llama-style decoder-only transformer.
 *
 * TEST INFRASTRUCTURE ONLY: the plain, slow, single-purpose CPU definition
 * that the HIP path is checked against.  Only tests, the smoke check and the
 * bench's CPU-baseline leg may load it.  It shares no code with the HIP
 * library.
 *
 * What it follows.  The paper (Kernel Looping, arXiv 2410.23668) names the
 * blocks of a token step (Sec. 2: Embedding, 32 x Decoder, Classifier,
 * Sampling) and the operators inside a decoder layer (Sec. 1 and Sec. 2:
 * GEMMs, RMSNorm, SiLU, SDPA with softmax), for BF16 Llama 3.1 models
 * (Table 1, Table 2).  It does not print the layer equations, so the layer
 * here is the standard Llama decoder layer, written out in its plain
 * definition:
 *   u = RMSNorm(x; g_attn)
 *   q = Wq u, k = Wk u, v = Wv u;  q, k rotated (RoPE) at the token position
 *   K[pos] = bf16(k), V[pos] = bf16(v)
 *   o_h = sum_j softmax_j(q_h . K[g(h)][j] / sqrt(d)) V[g(h)][j], j = 0..pos
 *   x = x + Wo o
 *   u = RMSNorm(x; g_ffn);  m = silu(Wg u) * (Wu u);  x = x + Wd m
 * and after L layers: logits = Wlm RMSNorm(x; g_final).
 * Readings taken where the paper is silent (each stated at its function):
 * half-split RoPE pairs, no rope scaling, post-RoPE cached keys, GQA by
 * contiguous head groups, the new k/v rounded to bf16 before attention,
 * epsilon inside the square root, untied embedding and LM head.
 *
 * Arithmetic is fp64 throughout (sums in index order); bf16 enters only as
 * the storage format of weights and the KV cache.  nthreads > 1 splits
 * independent output rows (GEMV rows, attention heads) across OpenMP threads,
 * which changes no sum's order, so results do not depend on thread count.
 *
 * Parity pins (the tests that tie this file to the mathematics) are in
 * tests/test_oracle_pins.py: bf16 rounding against a library conversion,
 * RMSNorm closed forms, one-hot GEMV columns, RoPE as complex rotation,
 * attention special cases (one key, zero query, two keys, GQA = repeated
 * MHA, permutation), SwiGLU closed forms, a zero-update whole step, and an
 * independent brute-force evaluation of small models.
 */
#include "kl_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ---- bf16 storage format ------------------------------------------------ */

/* bf16 is the upper half of an IEEE binary32: decode by a 16-bit shift. */
double klo_bf16_to_f64(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Round a double to the nearest bf16 value, ties to even, straight from the
 * double (no intermediate float rounding).  bf16 keeps 8 significant bits and
 * binary32's exponent range; below 2^-126 the spacing is fixed at 2^-133. */
uint16_t klo_f64_to_bf16(double v) {
    if (isnan(v)) return 0x7FC0;
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    double a = fabs(v);
    if (isinf(a)) return sign | 0x7F80;
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);                                  /* a = m 2^e, m in [0.5, 1) */
    int qexp = e - 8;                              /* spacing of 8-bit significands */
    if (qexp < -133) qexp = -133;
    double q = ldexp(1.0, qexp);
    double r = nearbyint(a / q) * q;               /* default rounding: ties to even */
    if (r >= ldexp(1.0, 128)) return sign | 0x7F80;
    float f = (float)r;                            /* exact: r has <= 8 significant bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return sign | (uint16_t)(u >> 16);
}

void klo_bf16_to_f64_array(const uint16_t *src, double *dst, int64_t n) {
    for (int64_t i = 0; i < n; ++i) dst[i] = klo_bf16_to_f64(src[i]);
}

void klo_f64_to_bf16_array(const double *src, uint16_t *dst, int64_t n) {
    for (int64_t i = 0; i < n; ++i) dst[i] = klo_f64_to_bf16(src[i]);
}

/* ---- operators --------------------------------------------------------- */

/* RMSNorm (named in Sec. 2): u_i = x_i / sqrt(mean_i(x_i^2) + eps) * g_i.
 * Reading: eps inside the square root, gain applied after normalising. */
void klo_rmsnorm(int32_t n, const double *x, const uint16_t *gain, double eps, double *u) {
    double ss = 0.0;
    for (int32_t i = 0; i < n; ++i) ss += x[i] * x[i];
    double r = 1.0 / sqrt(ss / (double)n + eps);
    for (int32_t i = 0; i < n; ++i) u[i] = x[i] * r * klo_bf16_to_f64(gain[i]);
}

/* GEMV (the decoder's GEMMs at batch 1, Sec. 2): y_j = sum_i W[j][i] u_i,
 * W in nn.Linear layout [rows = out][cols = in]. */
void klo_gemv(int32_t rows, int32_t cols, const uint16_t *w, const double *u, double *y,
              int32_t nthreads) {
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1)
    for (int32_t j = 0; j < rows; ++j) {
        const uint16_t *row = w + (int64_t)j * cols;
        double acc = 0.0;
        for (int32_t i = 0; i < cols; ++i) acc += klo_bf16_to_f64(row[i]) * u[i];
        y[j] = acc;
    }
}

/* Rotary position embedding of one head vector at position pos.
 * Reading (the paper does not define it): pairs (i, i + d/2) for i < d/2,
 * frequency w_i = theta^(-2i/d), angle pos * w_i, rotation
 *   (a, b) -> (a cos - b sin, a sin + b cos);  no frequency scaling. */
void klo_rope(int32_t head_dim, double theta, int32_t pos, double *y) {
    int32_t half = head_dim / 2;
    for (int32_t i = 0; i < half; ++i) {
        double w = pow(theta, -2.0 * (double)i / (double)head_dim);
        double phi = (double)pos * w;
        double c = cos(phi), s = sin(phi);
        double a = y[i], b = y[i + half];
        y[i] = a * c - b * s;
        y[i + half] = a * s + b * c;
    }
}

/* softmax (Sec. 1 names it among the decoder's streaming operators):
 * a_j = exp(s_j - max s) / sum_k exp(s_k - max s). */
void klo_softmax(int32_t n, const double *s, double *a) {
    double mx = -INFINITY;
    for (int32_t j = 0; j < n; ++j) if (s[j] > mx) mx = s[j];
    double sum = 0.0;
    for (int32_t j = 0; j < n; ++j) { a[j] = exp(s[j] - mx); sum += a[j]; }
    for (int32_t j = 0; j < n; ++j) a[j] /= sum;
}

/* SDPA over the KV cache for one sequence of one layer (Sec. 2 names SDPA).
 * q: [n_heads][d]; k_seq, v_seq: [n_kv][capacity][d] bf16; attends to slots
 * 0..pos (pos + 1 keys, no other mask).  Query head h reads KV head
 * g = h / (n_heads / n_kv) (contiguous groups).  Scores are scaled by
 * 1/sqrt(d). */
void klo_attention(int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, int32_t pos,
                   int32_t capacity, const double *q, const uint16_t *k_seq,
                   const uint16_t *v_seq, double *o) {
    int32_t n = pos + 1, group = n_heads / n_kv_heads;
    double scale = 1.0 / sqrt((double)head_dim);
    double *s = (double *)malloc(sizeof(double) * (size_t)n);
    double *a = (double *)malloc(sizeof(double) * (size_t)n);
    for (int32_t h = 0; h < n_heads; ++h) {
        int32_t g = h / group;
        const uint16_t *K = k_seq + (int64_t)g * capacity * head_dim;
        const uint16_t *V = v_seq + (int64_t)g * capacity * head_dim;
        const double *qh = q + (int64_t)h * head_dim;
        for (int32_t j = 0; j < n; ++j) {
            double dot = 0.0;
            for (int32_t i = 0; i < head_dim; ++i)
                dot += qh[i] * klo_bf16_to_f64(K[(int64_t)j * head_dim + i]);
            s[j] = dot * scale;
        }
        klo_softmax(n, s, a);
        double *oh = o + (int64_t)h * head_dim;
        for (int32_t i = 0; i < head_dim; ++i) oh[i] = 0.0;
        for (int32_t j = 0; j < n; ++j)
            for (int32_t i = 0; i < head_dim; ++i)
                oh[i] += a[j] * klo_bf16_to_f64(V[(int64_t)j * head_dim + i]);
    }
    free(s);
    free(a);
}

/* SwiGLU MLP activation (SiLU is named in Sec. 2): m_i = silu(g_i) * up_i,
 * silu(z) = z / (1 + exp(-z)). */
void klo_swiglu(int32_t n, const double *gate, const double *up, double *m) {
    for (int32_t i = 0; i < n; ++i) m[i] = gate[i] / (1.0 + exp(-gate[i])) * up[i];
}

/* Mixture-of-experts routing (the Mixtral entry of Table 2; the paper does
 * not describe the layer, the reading follows the model's definition): the
 * top_k largest router logits, taken one at a time as the largest not yet
 * taken with the lowest index winning a tie, weighted by the softmax of the
 * taken logits (equal to the softmax over all logits renormalised over the
 * taken ones). */
void klo_route(int32_t n, int32_t top_k, const double *logits, int32_t *idx, double *w) {
    for (int32_t k = 0; k < top_k; ++k) {
        int32_t best = -1;
        for (int32_t e = 0; e < n; ++e) {
            int32_t taken = 0;
            for (int32_t j = 0; j < k; ++j) taken |= idx[j] == e;
            if (!taken && (best < 0 || logits[e] > logits[best])) best = e;
        }
        idx[k] = best;
    }
    double s[8];
    for (int32_t k = 0; k < top_k; ++k) s[k] = logits[idx[k]];
    klo_softmax(top_k, s, w);
}

/* ---- one decode step ----------------------------------------------------- */

int32_t klo_decode_step(const klo_config *cfg, const uint16_t *embed,
                        const uint16_t *final_norm, const uint16_t *lm_head,
                        const klo_layer *layers, int32_t batch, const int32_t *tokens,
                        const int32_t *positions, uint16_t *kcache, uint16_t *vcache,
                        int32_t kv_batch, int32_t capacity, double *logits, double *hidden,
                        double *router, int32_t nthreads) {
    const int32_t L = cfg->n_layers, H = cfg->hidden, nq = cfg->n_heads,
                  nkv = cfg->n_kv_heads, d = cfg->head_dim, F = cfg->ffn_dim,
                  Vv = cfg->vocab;
    const int32_t E = cfg->n_experts > 1 ? cfg->n_experts : 1, K = cfg->top_k;
    if (E > 1 && (K < 1 || K > E || K > 8)) return -1;
    for (int32_t b = 0; b < batch; ++b) {
        if (tokens[b] < 0 || tokens[b] >= Vv) return -1;
        if (positions[b] < 0 || positions[b] >= capacity) return -1;
    }
    double *x = (double *)malloc(sizeof(double) * (size_t)H);
    double *u = (double *)malloc(sizeof(double) * (size_t)H);
    double *q = (double *)malloc(sizeof(double) * (size_t)nq * d);
    double *k = (double *)malloc(sizeof(double) * (size_t)nkv * d);
    double *v = (double *)malloc(sizeof(double) * (size_t)nkv * d);
    double *o = (double *)malloc(sizeof(double) * (size_t)nq * d);
    double *y = (double *)malloc(sizeof(double) * (size_t)(H > F ? H : F));
    double *gt = (double *)malloc(sizeof(double) * (size_t)F);
    double *up = (double *)malloc(sizeof(double) * (size_t)F);
    double *m = (double *)malloc(sizeof(double) * (size_t)F);
    double *acc = (double *)malloc(sizeof(double) * (size_t)H);
    double *rl = (double *)malloc(sizeof(double) * (size_t)E);
    const int64_t seq_stride = (int64_t)nkv * capacity * d;      /* one (layer, seq) block */

    for (int32_t b = 0; b < batch; ++b) {
        const int32_t t = tokens[b], p = positions[b];
        /* Embedding block (Sec. 2): the token's row, widened to fp64. */
        for (int32_t i = 0; i < H; ++i) x[i] = klo_bf16_to_f64(embed[(int64_t)t * H + i]);

        for (int32_t l = 0; l < L; ++l) {
            const klo_layer *W = &layers[l];
            uint16_t *Kl = kcache + ((int64_t)l * kv_batch + b) * seq_stride;
            uint16_t *Vl = vcache + ((int64_t)l * kv_batch + b) * seq_stride;

            klo_rmsnorm(H, x, W->attn_norm, cfg->rms_eps, u);
            klo_gemv(nq * d, H, W->wq, u, q, nthreads);
            klo_gemv(nkv * d, H, W->wk, u, k, nthreads);
            klo_gemv(nkv * d, H, W->wv, u, v, nthreads);
            /* Q/K/V biases where the model has them, before RoPE */
            if (W->bq)
                for (int32_t i = 0; i < nq * d; ++i) q[i] += klo_bf16_to_f64(W->bq[i]);
            if (W->bk)
                for (int32_t i = 0; i < nkv * d; ++i) k[i] += klo_bf16_to_f64(W->bk[i]);
            if (W->bv)
                for (int32_t i = 0; i < nkv * d; ++i) v[i] += klo_bf16_to_f64(W->bv[i]);
            for (int32_t h = 0; h < nq; ++h) klo_rope(d, cfg->rope_theta, p, q + (int64_t)h * d);
            for (int32_t g = 0; g < nkv; ++g) klo_rope(d, cfg->rope_theta, p, k + (int64_t)g * d);

            /* Reading: the cache holds post-RoPE keys; the new k and v are
             * stored as bf16 and attention reads them back like any slot. */
            for (int32_t g = 0; g < nkv; ++g)
                for (int32_t i = 0; i < d; ++i) {
                    Kl[((int64_t)g * capacity + p) * d + i] = klo_f64_to_bf16(k[(int64_t)g * d + i]);
                    Vl[((int64_t)g * capacity + p) * d + i] = klo_f64_to_bf16(v[(int64_t)g * d + i]);
                }
            klo_attention(nq, nkv, d, p, capacity, q, Kl, Vl, o);

            klo_gemv(H, nq * d, W->wo, o, y, nthreads);
            for (int32_t i = 0; i < H; ++i) x[i] += y[i];

            klo_rmsnorm(H, x, W->ffn_norm, cfg->rms_eps, u);
            if (E == 1) {
                klo_gemv(F, H, W->w_gate, u, gt, nthreads);
                klo_gemv(F, H, W->w_up, u, up, nthreads);
                klo_swiglu(F, gt, up, m);
                klo_gemv(H, F, W->w_down, m, y, nthreads);
                for (int32_t i = 0; i < H; ++i) x[i] += y[i];
            } else {
                /* mixture of experts: the router, then the weighted sum of
                 * the chosen experts' SwiGLU MLPs */
                int32_t idx[8];
                double w[8];
                klo_gemv(E, H, W->w_router, u, rl, nthreads);
                if (router) memcpy(router + ((int64_t)b * L + l) * E, rl, sizeof(double) * (size_t)E);
                klo_route(E, K, rl, idx, w);
                for (int32_t i = 0; i < H; ++i) acc[i] = 0.0;
                for (int32_t k = 0; k < K; ++k) {
                    const int64_t e = idx[k];
                    klo_gemv(F, H, W->w_gate + e * F * H, u, gt, nthreads);
                    klo_gemv(F, H, W->w_up + e * F * H, u, up, nthreads);
                    klo_swiglu(F, gt, up, m);
                    klo_gemv(H, F, W->w_down + e * H * F, m, y, nthreads);
                    for (int32_t i = 0; i < H; ++i) acc[i] += w[k] * y[i];
                }
                for (int32_t i = 0; i < H; ++i) x[i] += acc[i];
            }
        }
        if (hidden) memcpy(hidden + (int64_t)b * H, x, sizeof(double) * (size_t)H);
        /* Classifier block (Sec. 2): final RMSNorm, then the (untied) LM head. */
        klo_rmsnorm(H, x, final_norm, cfg->rms_eps, u);
        klo_gemv(Vv, H, lm_head, u, logits + (int64_t)b * Vv, nthreads);
    }
    free(x); free(u); free(q); free(k); free(v); free(o); free(y); free(gt); free(up); free(m);
    free(acc); free(rl);
    return 0;
}
