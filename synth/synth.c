/*
 * Seeded synthetic inputs shared by the tests, the bench and the oracle's
 * callers.  This module holds none of the decode step's arithmetic: it only
 * turns (seed, stream id, element index) into numbers.
 *
 * Generator (counter-based, so the result does not depend on thread count):
 *   key      = mix64(seed * G + mix64(stream_id + 1))
 *   word(i)  = mix64(key + (i + 1) * G)
 * where G = 0x9E3779B97F4A7C15 and mix64 is the SplitMix64 output function
 * (Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
 * OOPSLA 2014).  Uniforms take the top 53 bits of a word, mapped to (0, 1].
 * Normals use the Box-Muller transform in double on the word pair (2j, 2j+1):
 *   r = sqrt(-2 ln u0), n(2j) = r cos(2 pi u1), n(2j+1) = r sin(2 pi u1),
 * then mean + std * n is rounded to float and then to bfloat16 (round to
 * nearest, ties to even).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define SYN_GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t stream_id) {
    return mix64(seed * SYN_GOLDEN + mix64(stream_id + 1));
}

static inline uint64_t word_at(uint64_t key, uint64_t i) {
    return mix64(key + (i + 1) * SYN_GOLDEN);
}

/* (0, 1]: never 0, so log() below is finite. */
static inline double unit_open0(uint64_t w) {
    return (double)((w >> 11) + 1) * (1.0 / 9007199254740992.0);
}

static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u) {           /* inf / nan */
        return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
    }
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

uint64_t syn_word(uint64_t seed, uint64_t stream_id, uint64_t i) {
    return word_at(stream_key(seed, stream_id), i);
}

/* dst[i] for i in [0, n): bf16 of mean + std * N(0,1). */
void syn_normal_bf16(uint16_t *dst, int64_t n, uint64_t seed, uint64_t stream_id,
                     double mean, double std, int nthreads) {
    const uint64_t key = stream_key(seed, stream_id);
    const int64_t npairs = (n + 1) / 2;
    const double two_pi = 6.283185307179586476925286766559;
    (void)nthreads;
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t j = 0; j < npairs; ++j) {
        double u0 = unit_open0(word_at(key, (uint64_t)(2 * j)));
        double u1 = unit_open0(word_at(key, (uint64_t)(2 * j + 1)));
        double r = sqrt(-2.0 * log(u0));
        double a = two_pi * u1;
        double n0 = r * cos(a), n1 = r * sin(a);
        dst[2 * j] = f32_to_bf16_rne((float)(mean + std * n0));
        if (2 * j + 1 < n) dst[2 * j + 1] = f32_to_bf16_rne((float)(mean + std * n1));
    }
}

/* dst[i] uniform in [lo, hi) by multiply-shift of the word's top 32 bits. */
void syn_uniform_int32(int32_t *dst, int64_t n, uint64_t seed, uint64_t stream_id,
                       int32_t lo, int32_t hi) {
    const uint64_t key = stream_key(seed, stream_id);
    const uint64_t span = (uint64_t)((int64_t)hi - (int64_t)lo);
    for (int64_t i = 0; i < n; ++i) {
        uint64_t w = word_at(key, (uint64_t)i) >> 32;
        dst[i] = (int32_t)((int64_t)lo + (int64_t)((w * span) >> 32));
    }
}

/* dst[i] uniform in (0, 1] as double (used for the distribution tests). */
void syn_uniform_f64(double *dst, int64_t n, uint64_t seed, uint64_t stream_id) {
    const uint64_t key = stream_key(seed, stream_id);
    for (int64_t i = 0; i < n; ++i) dst[i] = unit_open0(word_at(key, (uint64_t)i));
}
