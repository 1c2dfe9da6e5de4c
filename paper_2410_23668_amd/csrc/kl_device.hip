// Device code of the decode step for gfx950 (CDNA4).
//
// One kernel, kl_step_kernel, runs any contiguous run of the step's phases:
//   embed | for each layer: qkv, attn, oproj, gateup, down | head
// The three schedules differ only in how many launches cover the run:
//   looped     one cooperative launch for everything (kernel looping, Sec. 2
//              and Sec. 3.2 of arXiv 2410.23668: the L chained layer calls
//              become one call with an outer loop; kernel boundaries become
//              device-scope grid barriers),
//   per-layer  one launch per layer (the fused-layer kernel K0 of Sec. 2),
//   per-op     one launch per phase.
// The work partition depends only on StepParams::nwg, so every schedule
// performs the same arithmetic in the same order: results are bit-identical.
//
// Weights are pre-packed into 1 KiB tiles of 8 rows x 64 columns (bf16,
// row-major inside the tile); the tiles of one 8-row group are contiguous
// along K.  A wave reads one tile per 16-byte-per-lane load: lane l holds row
// l/8, columns 8*(l%8) .. +7.  Activations are fp32 in LDS; accumulation is
// fp32 with a fixed order.

#include "kl_internal.h"
#include "kl.h"

namespace kl {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- helpers

__device__ __forceinline__ float bf_lo(unsigned u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(unsigned u) { return __uint_as_float(u & 0xffff0000u); }
__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float((unsigned)h << 16); }

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f2bf(float f) {
    unsigned u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                 CTRL, 0xF, 0xF, false));
}
// DPP controls: quad_perm [1,0,3,2] = 0xB1, [2,3,0,1] = 0x4E,
// row_half_mirror = 0x141, row_mirror = 0x140.
// Sum over aligned groups of 8 lanes; every lane of the group gets the sum.
__device__ __forceinline__ float sum8(float v) {
    v += dpp<0xB1>(v);
    v += dpp<0x4E>(v);
    v += dpp<0x141>(v);
    return v;
}
__device__ __forceinline__ float sum16(float v) { v = sum8(v); return v + dpp<0x140>(v); }

template <int LP>
__device__ __forceinline__ float sum_lanes(float v) {
    if constexpr (LP == 8) return sum8(v);
    else return sum16(v);
}

__device__ __forceinline__ float wave_sum(float v) {
    v = sum16(v);
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
    for (int off = 1; off < 64; off <<= 1) v = fmaxf(v, __shfl_xor(v, off));
    return v;
}

// Sum over the workgroup; every thread gets the same value (fixed order).
__device__ __forceinline__ float block_sum(float v, float *sm) {
    v = wave_sum(v);
    const int wid = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) sm[wid] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t += sm[w];
    __syncthreads();
    return t;
}

__device__ __forceinline__ void split_range(int n, int parts, int i, int &a, int &b) {
    a = (int)((long long)n * i / parts);
    b = (int)((long long)n * (i + 1) / parts);
}

__device__ __forceinline__ int eff_pos(const StepParams &P, int b) {
    const int p = P.positions[b];
    const int lim = min(P.cap, P.max_seq);
    return p < 0 ? 0 : (p >= lim ? lim - 1 : p);
}
__device__ __forceinline__ int eff_tok(const StepParams &P, int b) {
    const int t = P.tokens[b];
    return (t < 0 || t >= P.V) ? 0 : t;
}

__device__ __forceinline__ size_t kv_row(const StepParams &P, int l, int b, int g) {
    return (((size_t)l * P.kv_batch + b) * P.nkv + g) * (size_t)P.cap;
}

// ---------------------------------------------------------------- grid barrier
//
// A generation barrier over the nwg co-resident workgroups.  Arrivals count
// up one word; the last arrival resets it and bumps the generation word that
// the others poll.  Release/acquire at agent scope makes every workgroup's
// global writes before the barrier visible to every workgroup after it,
// across XCDs.  The wait is bounded: after ~2 s it raises KL_DEVERR_BARRIER,
// and any later wait returns at once once that bit is set, so a broken
// barrier ends the kernel instead of hanging it.
constexpr long long kBarrierTicks = 200000000LL;   // s_memrealtime runs at 100 MHz

__device__ __forceinline__ void grid_sync(const StepParams &P) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned *arrive = P.bar;
        unsigned *gen = P.bar + 64;
        const unsigned g0 = __hip_atomic_load(gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const unsigned old = __hip_atomic_fetch_add(arrive, 1u, __ATOMIC_ACQ_REL,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        if (old == (unsigned)P.nwg - 1u) {
            __hip_atomic_store(arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_fetch_add(gen, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            const long long t0 = wall_clock64();
            while (__hip_atomic_load(gen, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) == g0) {
                if (__hip_atomic_load(P.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) &
                    KL_DEVERR_BARRIER)
                    break;
                if (wall_clock64() - t0 > kBarrierTicks) {
                    __hip_atomic_fetch_or(P.err, KL_DEVERR_BARRIER, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
    }
    __syncthreads();
}

// ---------------------------------------------------------------- params
//
// Each phase is a separate (non-inlined) function that reads the step
// parameters from the kernel-argument segment itself.  Inlining all phases
// into the layer loop would let the compiler hoist every phase's address
// arithmetic out of the loop and keep it live across all phases, which
// exhausts registers; separate functions keep each phase's registers local.
// The kernel passes the address of its argument segment down as an integer
// (the segment-pointer builtin is only valid inside the kernel itself), and
// the callee makes it wave-uniform again so the fields load with s_load.
#define KL_KARG __attribute__((address_space(4)))

typedef uint64_t KArg;

__device__ __forceinline__ KArg kernarg_address() {
#if defined(__HIP_DEVICE_COMPILE__)
    return (KArg)(const KL_KARG char *)__builtin_amdgcn_kernarg_segment_ptr();
#else
    return 0;
#endif
}

__device__ __forceinline__ StepParams load_params(KArg ka) {
#if defined(__HIP_DEVICE_COMPILE__)
    const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)ka);
    const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(ka >> 32));
    const KL_KARG StepParams *p = (const KL_KARG StepParams *)(((KArg)hi << 32) | lo);
    return *p;
#else
    return StepParams{};   // the host pass only type-checks device code
#endif
}

extern __shared__ __align__(16) char kl_smem[];

// ---------------------------------------------------------------- LDS layout

struct Lds {
    float *a;     // activation vector (max K extent), or the attention area
    float *red;   // [kWaves][kRgBatch][kTileRows] GEMV partial sums
    float *sm;    // small reductions and flags
};

__device__ __forceinline__ Lds lds_layout(char *smem, const StepParams &P) {
    Lds s;
    int amax = max(max(P.Hp, P.Ap), P.Fp);
    const int attn = P.group * P.d + P.group * kAttnSub + P.group * 4 + kWaves * P.group * P.d;
    amax = max(amax, attn);
    amax = (amax + 63) & ~63;
    s.a = reinterpret_cast<float *>(smem);
    s.red = s.a + amax;
    s.sm = s.red + kWaves * kRgBatch * kTileRows;
    return s;
}

// ---------------------------------------------------------------- activations

// a[i] = x[i] * rsqrt(mean(x^2) + eps) * gain[i] for i < n, 0 up to npad.
__device__ __forceinline__ void rmsnorm_to_lds(const float *__restrict__ x, const float *__restrict__ gain,
                               int n, int npad, float eps, float *a, float *sm) {
    float ss = 0.f;
    for (int i = threadIdx.x; i < n; i += kThreads) {
        const float v = x[i];
        ss = fmaf(v, v, ss);
    }
    ss = block_sum(ss, sm);
    const float r = 1.0f / sqrtf(ss / (float)n + eps);
    for (int i = threadIdx.x; i < npad; i += kThreads) a[i] = (i < n) ? x[i] * r * gain[i] : 0.f;
    __syncthreads();
}

__device__ __forceinline__ void vec_to_lds(const float *__restrict__ src, int n, float *a) {
    for (int i = threadIdx.x; i < n; i += kThreads) a[i] = src[i];
    __syncthreads();
}

// ---------------------------------------------------------------- GEMV engine
//
// y[r] = sum_k W[r][k] a[k] for the rows of row groups [rg0, rg1) of a packed
// matrix with KT k-tiles per row group.  Each wave takes a fixed slice of the
// k-tiles of every row group (split-K inside the workgroup), keeps U tile
// loads in flight, and reduces its partial dot products over the 8 lanes of a
// row with DPP.  The slices are summed in wave order through LDS, and epi is
// called once per row pair (r even, r + 1).
template <class Epi>
__device__ __forceinline__ void gemv_rows(const uint8_t *__restrict__ W, int KT, int rg0, int rg1,
                                          const float *__restrict__ a, float *red, Epi &&epi) {
    constexpr int U = 8;
    // wave-uniform values live in scalar registers, so every branch below is
    // a scalar branch and the loads of the main loop are unconditional
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int kt0 = (wid * KT) / kWaves, kt1 = ((wid + 1) * KT) / kWaves;
    const int nk = kt1 - kt0;
    const int row = lane >> 3, sub = lane & 7;
    const uint8_t *base = W + (size_t)lane * 16;
    const float *abase = a + sub * 8;
    for (int rb0 = rg0; rb0 < rg1; rb0 += kRgBatch) {
        const int nrg = min(kRgBatch, rg1 - rb0);
        const int n = nk * nrg;
        if (n > 0) {
            u32x4 buf[U];
            int lr = 0, lk = 0;        // next tile to load
            int cr = 0, ck = 0;        // next tile to consume
            float acc = 0.f;
            auto load_next = [&]() {
                const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(
                    base + ((size_t)(rb0 + lr) * KT + kt0 + lk) * kTileBytes));
                if (++lk == nk) { lk = 0; ++lr; }
                return v;
            };
            auto consume = [&](const u32x4 wv) {
                const float *ap = abase + (kt0 + ck) * kTileK;
                const float4 a0 = *reinterpret_cast<const float4 *>(ap);
                const float4 a1 = *reinterpret_cast<const float4 *>(ap + 4);
                acc = fmaf(bf_lo(wv.x), a0.x, acc);
                acc = fmaf(bf_hi(wv.x), a0.y, acc);
                acc = fmaf(bf_lo(wv.y), a0.z, acc);
                acc = fmaf(bf_hi(wv.y), a0.w, acc);
                acc = fmaf(bf_lo(wv.z), a1.x, acc);
                acc = fmaf(bf_hi(wv.z), a1.y, acc);
                acc = fmaf(bf_lo(wv.w), a1.z, acc);
                acc = fmaf(bf_hi(wv.w), a1.w, acc);
                if (++ck == nk) {
                    const float t = sum8(acc);
                    if (sub == 0) red[(wid * kRgBatch + cr) * kTileRows + row] = t;
                    acc = 0.f;
                    ck = 0;
                    ++cr;
                }
            };
            if (n >= U) {
                // every path into the main loop has exactly U loads in flight, so
                // the compiler can wait for the oldest one only (vmcnt(U-1))
#pragma unroll
                for (int s = 0; s < U; ++s) buf[s] = load_next();
                int i0 = 0;
                for (; i0 + 2 * U <= n; i0 += U) {
#pragma unroll
                    for (int s = 0; s < U; ++s) {
                        // consume before refilling: the refill reuses the slot's registers
                        consume(buf[s]);
                        buf[s] = load_next();
                    }
                }
                const int rem = n - i0;   // in [U, 2U): U items in buf, rem - U still to load
#pragma unroll
                for (int s = 0; s < U; ++s) {
                    consume(buf[s]);
                    if (s + U < rem) buf[s] = load_next();
                }
#pragma unroll
                for (int s = 0; s < U; ++s)
                    if (s + U < rem) consume(buf[s]);
            } else {
#pragma unroll
                for (int s = 0; s < U; ++s)
                    if (s < n) buf[s] = load_next();
#pragma unroll
                for (int s = 0; s < U; ++s)
                    if (s < n) consume(buf[s]);
            }
        }
        __syncthreads();
        for (int t = threadIdx.x; t < nrg * (kTileRows / 2); t += kThreads) {
            const int rgi = t / (kTileRows / 2), pr = (t % (kTileRows / 2)) * 2;
            float y0 = 0.f, y1 = 0.f;
            for (int w = 0; w < kWaves; ++w) {
                if (((w + 1) * KT) / kWaves == (w * KT) / kWaves) continue;   // empty slice
                y0 += red[(w * kRgBatch + rgi) * kTileRows + pr];
                y1 += red[(w * kRgBatch + rgi) * kTileRows + pr + 1];
            }
            epi((rb0 + rgi) * kTileRows + pr, y0, y1);
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------- phases

// Embedding block (Sec. 2): x = f32(E[token]).  Workgroup 0 records bad
// token ids and positions in the device error word.
__device__ __noinline__ void phase_embed(KArg ka) {
    const StepParams P = load_params(ka);
    if (blockIdx.x == 0) {
        for (int b = threadIdx.x; b < P.B; b += kThreads) {
            const int t = P.tokens[b], p = P.positions[b];
            int bits = 0;
            if (t < 0 || t >= P.V) bits |= KL_DEVERR_TOKEN;
            if (p < 0 || p >= P.cap || p >= P.max_seq) bits |= KL_DEVERR_POSITION;
            if (bits) atomicOr(P.err, bits);
        }
    }
    const int total = P.B * P.Hp;
    for (int idx = blockIdx.x * kThreads + threadIdx.x; idx < total; idx += P.nwg * kThreads) {
        const int b = idx / P.Hp, i = idx % P.Hp;
        P.x[idx] = (i < P.H) ? bf2f(P.embed[(size_t)eff_tok(P, b) * P.H + i]) : 0.f;
    }
}

// RMSNorm + fused Q/K/V projection + RoPE + KV-cache append.  Q/K rows are
// packed in rotation pairs (dims i and i + d/2 adjacent), V rows in order.
__device__ __noinline__ void phase_qkv(KArg ka, int l) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    int rg0, rg1;
    split_range(P.qkv_rg, P.nwg, blockIdx.x, rg0, rg1);
    if (rg0 == rg1) return;
    const uint8_t *Lb = P.arena + (size_t)l * P.layer_stride;
    const float *gain = reinterpret_cast<const float *>(Lb + P.off_attn_norm);
    const int d = P.d, half = P.d / 2, qd = P.nq * P.d, kd = P.nkv * P.d;
    for (int b = 0; b < P.B; ++b) {
        rmsnorm_to_lds(P.x + (size_t)b * P.Hp, gain, P.H, P.Hp, P.eps, S.a, S.sm);
        const int p = eff_pos(P, b);
        const float2 *rp = P.rope + (size_t)p * half;
        gemv_rows(Lb + P.off_qkv, P.Hp / kTileK, rg0, rg1, S.a, S.red,
                  [&](int r, float y0, float y1) {
                      if (r < qd + kd) {
                          const int h = r / d, i = (r % d) >> 1;
                          const float2 cs = rp[i];
                          const float u0 = y0 * cs.x - y1 * cs.y;
                          const float u1 = y0 * cs.y + y1 * cs.x;
                          if (r < qd) {
                              float *qq = P.q + (size_t)b * qd + (size_t)h * d;
                              qq[i] = u0;
                              qq[i + half] = u1;
                          } else {
                              uint16_t *kk = P.kc + (kv_row(P, l, b, h - P.nq) + p) * d;
                              kk[i] = f2bf(u0);
                              kk[i + half] = f2bf(u1);
                          }
                      } else {
                          const int rr = r - qd - kd, g = rr / d, j = rr % d;
                          uint16_t *vv = P.vc + (kv_row(P, l, b, g) + p) * d;
                          vv[j] = f2bf(y0);
                          vv[j + 1] = f2bf(y1);
                      }
                  });
    }
}

// One attention work item: the positions of chunk c of sequence b against KV
// head g, for the G query heads of that group.  Scores and probabilities are
// fp32; the chunk result is (running max, running sum, unnormalised output)
// per head.  The last workgroup to finish a (b, g) combines all chunks in
// chunk order and writes o.
template <int D, int G>
__device__ __noinline__ void attn_item(KArg ka, int l, int b, int g, int c) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    constexpr int LP = D / 8;                       // lanes per position
    constexpr int PP = 64 / LP;                     // positions per wave load
    constexpr int NG = kAttnSub / PP / kWaves;      // loads per wave per sub-chunk
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int pi = lane / LP, ds = (lane % LP) * 8;
    const int n = eff_pos(P, b) + 1;
    const int cs = (n + P.C - 1) / P.C;
    const int j0 = min(n, c * cs), j1 = min(n, j0 + cs);

    float *qs = S.a;                    // [G][D]
    float *sp = qs + G * D;             // [G][kAttnSub]
    float *st = sp + G * kAttnSub;      // [G][4]
    float *red = st + G * 4;            // [kWaves][G][D]
    const size_t row0 = kv_row(P, l, b, g);
    const uint16_t *Kb = P.kc + row0 * D;
    const uint16_t *Vb = P.vc + row0 * D;
    const float scale = 1.0f / sqrtf((float)D);

    for (int t = threadIdx.x; t < G * D; t += kThreads)
        qs[t] = P.q[(size_t)b * P.nq * D + (size_t)g * G * D + t];
    if (threadIdx.x < G) {
        st[threadIdx.x * 4 + 0] = -INFINITY;
        st[threadIdx.x * 4 + 1] = 0.f;
    }
    __syncthreads();
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;

    for (int js = j0; js < j1; js += kAttnSub) {
        const int len = min(kAttnSub, j1 - js);
        u32x4 kv[NG];
#pragma unroll
        for (int t = 0; t < NG; ++t) {
            const int jl = (wid * NG + t) * PP + pi;
            kv[t] = (jl < len) ? __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(
                                     Kb + (size_t)(js + jl) * D + ds))
                               : u32x4{0u, 0u, 0u, 0u};
        }
        // scores (q is read from LDS; all lanes take part in the lane sums)
#pragma unroll
        for (int t = 0; t < NG; ++t) {
            const int jl = (wid * NG + t) * PP + pi;
            const float kf[8] = {bf_lo(kv[t].x), bf_hi(kv[t].x), bf_lo(kv[t].y), bf_hi(kv[t].y),
                                 bf_lo(kv[t].z), bf_hi(kv[t].z), bf_lo(kv[t].w), bf_hi(kv[t].w)};
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float4 q0 = *reinterpret_cast<const float4 *>(qs + h * D + ds);
                const float4 q1 = *reinterpret_cast<const float4 *>(qs + h * D + ds + 4);
                float s = 0.f;
                s = fmaf(q0.x, kf[0], s);
                s = fmaf(q0.y, kf[1], s);
                s = fmaf(q0.z, kf[2], s);
                s = fmaf(q0.w, kf[3], s);
                s = fmaf(q1.x, kf[4], s);
                s = fmaf(q1.y, kf[5], s);
                s = fmaf(q1.z, kf[6], s);
                s = fmaf(q1.w, kf[7], s);
                s = sum_lanes<LP>(s);
                if (jl < len && (lane % LP) == 0) sp[h * kAttnSub + jl] = s * scale;
            }
        }
        // V loads go out now and land during the softmax step
#pragma unroll
        for (int t = 0; t < NG; ++t) {
            const int jl = (wid * NG + t) * PP + pi;
            kv[t] = (jl < len) ? __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(
                                     Vb + (size_t)(js + jl) * D + ds))
                               : u32x4{0u, 0u, 0u, 0u};
        }
        __syncthreads();
        // softmax statistics: wave h owns head h
        if (wid < G) {
            const int h = wid;
            float mx = -INFINITY;
            for (int j = lane; j < len; j += 64) mx = fmaxf(mx, sp[h * kAttnSub + j]);
            mx = wave_max(mx);
            const float mold = st[h * 4], mnew = fmaxf(mold, mx);
            const float resc = (mold == -INFINITY) ? 0.f : expf(mold - mnew);
            float sum = 0.f;
            for (int j = lane; j < len; j += 64) {
                const float e = expf(sp[h * kAttnSub + j] - mnew);
                sp[h * kAttnSub + j] = e;
                sum += e;
            }
            sum = wave_sum(sum);
            if (lane == 0) {
                st[h * 4 + 0] = mnew;
                st[h * 4 + 1] = st[h * 4 + 1] * resc + sum;
                st[h * 4 + 2] = resc;
            }
        }
        __syncthreads();
        // values
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float r = st[h * 4 + 2];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[h][e] *= r;
        }
#pragma unroll
        for (int t = 0; t < NG; ++t) {
            const int jl = (wid * NG + t) * PP + pi;
            if (jl < len) {
                const float vf[8] = {bf_lo(kv[t].x), bf_hi(kv[t].x), bf_lo(kv[t].y),
                                     bf_hi(kv[t].y), bf_lo(kv[t].z), bf_hi(kv[t].z),
                                     bf_lo(kv[t].w), bf_hi(kv[t].w)};
#pragma unroll
                for (int h = 0; h < G; ++h) {
                    const float pr = sp[h * kAttnSub + jl];
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pr, vf[e], acc[h][e]);
                }
            }
        }
        __syncthreads();
    }
    // reduce the PP position slots of each wave, then the waves in order
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float v = acc[h][e];
#pragma unroll
            for (int off = LP; off < 64; off <<= 1) v += __shfl_xor(v, off);
            acc[h][e] = v;
        }
    if (pi == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) red[(wid * G + h) * D + ds + e] = acc[h][e];
    }
    __syncthreads();
    float *part_bg = P.part + (size_t)(b * P.nkv + g) * P.C * G * (D + 2);
    float *out = part_bg + (size_t)c * G * (D + 2);
    for (int t = threadIdx.x; t < G * D; t += kThreads) {
        const int h = t / D, dd = t % D;
        float s = 0.f;
        for (int w = 0; w < kWaves; ++w) s += red[(w * G + h) * D + dd];
        out[h * (D + 2) + dd] = s;
    }
    if (threadIdx.x < G) {
        out[threadIdx.x * (D + 2) + D] = st[threadIdx.x * 4 + 0];
        out[threadIdx.x * (D + 2) + D + 1] = st[threadIdx.x * 4 + 1];
    }
    // publish this chunk; the last arrival for (b, g) combines
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    int *flag = reinterpret_cast<int *>(S.sm);
    if (threadIdx.x == 0) {
        unsigned *cnt = P.cnt + b * P.nkv + g;
        const unsigned old = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_ACQ_REL,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        const int last = old == (unsigned)(P.C - 1);
        if (last) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        flag[0] = last;
    }
    __syncthreads();
    if (flag[0]) {
        for (int t = threadIdx.x; t < G * D; t += kThreads) {
            const int h = t / D, dd = t % D;
            float M = -INFINITY;
            for (int cc = 0; cc < P.C; ++cc) M = fmaxf(M, part_bg[((size_t)cc * G + h) * (D + 2) + D]);
            float lsum = 0.f, num = 0.f;
            for (int cc = 0; cc < P.C; ++cc) {
                const float *pc = part_bg + ((size_t)cc * G + h) * (D + 2);
                const float mc = pc[D];
                if (mc == -INFINITY) continue;
                const float w = expf(mc - M);
                lsum = fmaf(pc[D + 1], w, lsum);
                num = fmaf(pc[dd], w, num);
            }
            P.o[(size_t)b * P.Ap + (size_t)(g * G + h) * D + dd] = num / lsum;
        }
    }
    __syncthreads();
}

template <int D>
__device__ __forceinline__ void attn_dispatch_g(KArg ka, int group, int l, int b, int g, int c) {
    switch (group) {
        case 1: attn_item<D, 1>(ka, l, b, g, c); break;
        case 2: attn_item<D, 2>(ka, l, b, g, c); break;
        case 4: attn_item<D, 4>(ka, l, b, g, c); break;
        default: attn_item<D, 8>(ka, l, b, g, c); break;
    }
}

__device__ __noinline__ void phase_attn(KArg ka, int l) {
    const StepParams P = load_params(ka);
    const int items = P.B * P.nkv * P.C;
    for (int it = blockIdx.x; it < items; it += P.nwg) {
        const int c = it % P.C, bg = it / P.C, g = bg % P.nkv, b = bg / P.nkv;
        if (P.d == 64) attn_dispatch_g<64>(ka, P.group, l, b, g, c);
        else attn_dispatch_g<128>(ka, P.group, l, b, g, c);
    }
}

// O projection + residual: x += Wo o (each row has one owner; no atomics).
__device__ __noinline__ void phase_oproj(KArg ka, int l) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    int rg0, rg1;
    split_range(P.o_rg, P.nwg, blockIdx.x, rg0, rg1);
    if (rg0 == rg1) return;
    const uint8_t *Lb = P.arena + (size_t)l * P.layer_stride;
    for (int b = 0; b < P.B; ++b) {
        vec_to_lds(P.o + (size_t)b * P.Ap, P.Ap, S.a);
        float *x = P.x + (size_t)b * P.Hp;
        gemv_rows(Lb + P.off_o, P.Ap / kTileK, rg0, rg1, S.a, S.red,
                  [&](int r, float y0, float y1) {
                      x[r] += y0;
                      x[r + 1] += y1;
                  });
    }
}

// RMSNorm + fused gate/up projection + SwiGLU: m = silu(Wg u) * (Wu u).
// Packed rows alternate gate i, up i.
__device__ __noinline__ void phase_gateup(KArg ka, int l) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    int rg0, rg1;
    split_range(P.gu_rg, P.nwg, blockIdx.x, rg0, rg1);
    if (rg0 == rg1) return;
    const uint8_t *Lb = P.arena + (size_t)l * P.layer_stride;
    const float *gain = reinterpret_cast<const float *>(Lb + P.off_ffn_norm);
    for (int b = 0; b < P.B; ++b) {
        rmsnorm_to_lds(P.x + (size_t)b * P.Hp, gain, P.H, P.Hp, P.eps, S.a, S.sm);
        float *m = P.m + (size_t)b * P.Fp;
        gemv_rows(Lb + P.off_gu, P.Hp / kTileK, rg0, rg1, S.a, S.red,
                  [&](int r, float g, float u) { m[r >> 1] = g / (1.0f + expf(-g)) * u; });
    }
}

// Down projection + residual: x += Wd m.
__device__ __noinline__ void phase_down(KArg ka, int l) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    int rg0, rg1;
    split_range(P.down_rg, P.nwg, blockIdx.x, rg0, rg1);
    if (rg0 == rg1) return;
    const uint8_t *Lb = P.arena + (size_t)l * P.layer_stride;
    for (int b = 0; b < P.B; ++b) {
        vec_to_lds(P.m + (size_t)b * P.Fp, P.Fp, S.a);
        float *x = P.x + (size_t)b * P.Hp;
        gemv_rows(Lb + P.off_down, P.Fp / kTileK, rg0, rg1, S.a, S.red,
                  [&](int r, float y0, float y1) {
                      x[r] += y0;
                      x[r + 1] += y1;
                  });
    }
}

// Classifier block (Sec. 2): final RMSNorm + LM head -> fp32 logits.
__device__ __noinline__ void phase_head(KArg ka) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    if (blockIdx.x == 0 && P.hidden_out) {
        for (int idx = threadIdx.x; idx < P.B * P.H; idx += kThreads)
            P.hidden_out[idx] = P.x[(size_t)(idx / P.H) * P.Hp + idx % P.H];
    }
    int rg0, rg1;
    split_range(P.head_rg, P.nwg, blockIdx.x, rg0, rg1);
    if (rg0 == rg1) return;
    for (int b = 0; b < P.B; ++b) {
        rmsnorm_to_lds(P.x + (size_t)b * P.Hp, P.final_norm, P.H, P.Hp, P.eps, S.a, S.sm);
        float *lg = P.logits + (size_t)b * P.V;
        const int V = P.V;
        gemv_rows(reinterpret_cast<const uint8_t *>(P.lm_head), P.Hp / kTileK, rg0, rg1, S.a, S.red, [&](int r, float y0, float y1) {
            if (r < V) lg[r] = y0;
            if (r + 1 < V) lg[r + 1] = y1;
        });
    }
}

// ---------------------------------------------------------------- kernels

__global__ __launch_bounds__(kThreads) void kl_step_kernel(StepParams P, int l0, int l1,
                                                          int phases) {
    const KArg ka = kernarg_address();
    bool started = false;
    auto next = [&]() {
        if (started) grid_sync(P);
        started = true;
    };
    if (phases & kPhEmbed) { next(); phase_embed(ka); }
    for (int l = l0; l < l1; ++l) {
        if (phases & kPhQkv) { next(); phase_qkv(ka, l); }
        if (phases & kPhAttn) { next(); phase_attn(ka, l); }
        if (phases & kPhOproj) { next(); phase_oproj(ka, l); }
        if (phases & kPhGateUp) { next(); phase_gateup(ka, l); }
        if (phases & kPhDown) { next(); phase_down(ka, l); }
    }
    if (phases & kPhHead) { next(); phase_head(ka); }
}

// Repack row-major bf16 matrices into 8x64 tiles.  rowmap[packed row] =
// (source id << 28) | source row, or -1 for a zero row; columns >= K are zero.
__global__ void kl_pack_rows_kernel(uint16_t *__restrict__ dst, int n_rg, int KT, int K,
                                    const int32_t *__restrict__ rowmap,
                                    const uint16_t *__restrict__ s0,
                                    const uint16_t *__restrict__ s1,
                                    const uint16_t *__restrict__ s2) {
    const size_t chunks = (size_t)n_rg * KT * 64;
    for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < chunks;
         idx += (size_t)gridDim.x * blockDim.x) {
        const int lane = (int)(idx % 64);
        const size_t tile = idx / 64;
        const int kt = (int)(tile % KT), rg = (int)(tile / KT);
        const int pr = rg * kTileRows + lane / 8, k = kt * kTileK + (lane % 8) * 8;
        const int m = rowmap[pr];
        unsigned w[4] = {0u, 0u, 0u, 0u};
        if (m >= 0) {
            const int sid = m >> 28, row = m & 0x0fffffff;
            const uint16_t *src = (sid == 0 ? s0 : (sid == 1 ? s1 : s2)) + (size_t)row * K;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const unsigned v = (k + e < K) ? src[k + e] : 0u;
                w[e >> 1] |= v << (16 * (e & 1));
            }
        }
        reinterpret_cast<u32x4 *>(dst)[idx] = u32x4{w[0], w[1], w[2], w[3]};
    }
}

__global__ void kl_gain_to_f32_kernel(float *dst, const uint16_t *src, int n, int npad) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < npad; i += gridDim.x * blockDim.x)
        dst[i] = (i < n) ? bf2f(src[i]) : 0.f;
}

// ---------------------------------------------------------------- launchers

hipError_t step_kernel_setup(int lds_bytes, int *max_blocks_per_cu) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kl_step_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (e != hipSuccess) return e;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(max_blocks_per_cu, kl_step_kernel,
                                                         kThreads, lds_bytes);
}

hipError_t launch_step(const StepParams &p, int first_layer, int last_layer, int phases,
                       bool cooperative, int lds_bytes, hipStream_t stream) {
    StepParams pc = p;
    if (cooperative) {
        void *args[] = {&pc, &first_layer, &last_layer, &phases};
        return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(kl_step_kernel),
                                          dim3(p.nwg), dim3(kThreads), args, lds_bytes, stream);
    }
    hipLaunchKernelGGL(kl_step_kernel, dim3(p.nwg), dim3(kThreads), lds_bytes, stream, pc,
                       first_layer, last_layer, phases);
    return hipGetLastError();
}

hipError_t launch_pack_rows(uint16_t *dst, int n_rg, int kt, int K, const int32_t *rowmap,
                            const uint16_t *src0, const uint16_t *src1, const uint16_t *src2,
                            hipStream_t stream) {
    const size_t chunks = (size_t)n_rg * kt * 64;
    const int blocks = (int)std::min<size_t>((chunks + 255) / 256, 65536);
    hipLaunchKernelGGL(kl_pack_rows_kernel, dim3(blocks), dim3(256), 0, stream, dst, n_rg, kt, K,
                       rowmap, src0, src1, src2);
    return hipGetLastError();
}

hipError_t launch_gain_to_f32(float *dst, const uint16_t *src, int n, int npad,
                              hipStream_t stream) {
    const int blocks = (npad + 255) / 256;
    hipLaunchKernelGGL(kl_gain_to_f32_kernel, dim3(blocks), dim3(256), 0, stream, dst, src, n,
                       npad);
    return hipGetLastError();
}

}  // namespace kl
