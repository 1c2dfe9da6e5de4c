// Device code of the decode step for gfx950 (CDNA4), included by the
// translation units that instantiate the step kernel (kl_step_*.hip).
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
// Pipelining across phases (the "pipelined outer loop" of Sec. 3.2): a phase
// issues the first loads of its weight tiles before it waits for the barrier
// that publishes its input activations, so HBM keeps streaming while the
// grid synchronises.  Data that crosses workgroups (activations, partials,
// the new KV slot) is written and read with device-coherent (agent-scope)
// accesses, so a barrier needs no cache write-back or invalidation: only the
// completion of the stores before the arrival.
//
// Weights are pre-packed into 1 KiB tiles of 8 rows x 64 columns (bf16,
// row-major inside the tile); the tiles of one 8-row group are contiguous
// along K.  A wave reads one tile per 16-byte-per-lane load: lane l holds row
// l/8, columns 8*(l%8) .. +7.  Activations are fp32 in LDS; accumulation is
// fp32 with a fixed order.

#pragma once

#include <type_traits>

#include "kl_internal.h"
#include "kl.h"

namespace kl {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- helpers

// The thread's index in its workgroup, opaque to the compiler at each use:
// values derived from it are formed where they are used instead of being
// hoisted out of the layer loop and kept live (or spilled) across the kernel.
__device__ __forceinline__ unsigned kl_tid() {
    unsigned t = __builtin_amdgcn_workitem_id_x();
    asm volatile("" : "+v"(t));
    return t;
}

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

// The two bf16 terms of a matrix-core activation: hi = bf16(x), lo =
// bf16(x - hi) (x - hi is exact in fp32), so hi + lo = x (1 + O(2^-17)).
// Two values per call, packed as (x0 | x1 << 16).
__device__ __forceinline__ void split_bf16x2(float x0, float x1, unsigned &hi, unsigned &lo) {
    const uint16_t h0 = f2bf(x0), h1 = f2bf(x1);
    hi = (unsigned)h0 | ((unsigned)h1 << 16);
    lo = (unsigned)f2bf(x0 - bf2f(h0)) | ((unsigned)f2bf(x1 - bf2f(h1)) << 16);
}
__device__ __forceinline__ void split_bf16(float x, uint16_t &hi, uint16_t &lo) {
    hi = f2bf(x);
    lo = f2bf(x - bf2f(hi));
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
    const int wid = kl_tid() >> 6;
    if ((kl_tid() & 63) == 0) sm[wid] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) t += sm[w];
    __syncthreads();
    return t;
}

__device__ __forceinline__ void split_range(int n, int parts, int i, int &a, int &b) {
    a = (int)((long long)n * i / parts);
    b = (int)((long long)n * (i + 1) / parts);
}

// A sequence whose token or position is out of range still runs through the
// step with clamped values (every read stays in bounds), but writes nothing
// the caller owns except NaN logits and hidden state: its K/V slots are left
// untouched.  The embedding phase raises the matching error bits.
// Greedy sampling (the Sampling block, Sec. 2, Fig. 3) reduces each
// candidate logit to a 64-bit key, (order-preserving bits of the logit << 32)
// | (0xFFFFFFFF - index): the largest key is the largest logit and, among equal
// logits, the lowest index.  NaN logits (a skipped sequence) are no
// candidates; key 0 means none and decodes to token -1 (out of range).
__device__ __forceinline__ unsigned long long argmax_key(float v, int idx) {
    const unsigned u = __float_as_uint(v);
    const unsigned ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((unsigned long long)ord << 32) | (0xFFFFFFFFu - (unsigned)idx);
}
__device__ __forceinline__ int key_token(unsigned long long k) {
    return k ? (int)(0xFFFFFFFFu - (unsigned)k) : -1;
}
__device__ __forceinline__ int raw_tok(const StepParams &P, int b) {
    if (P.tok_keys)
        return key_token(__hip_atomic_load(const_cast<unsigned long long *>(P.tok_keys + b),
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    return P.tokens[b];
}
__device__ __forceinline__ int raw_pos(const StepParams &P, int b) {
    return P.positions[b] + P.pos_add;
}

__device__ __forceinline__ int eff_pos(const StepParams &P, int b) {
    const int p = raw_pos(P, b);
    const int lim = min(P.cap, P.max_seq);
    return p < 0 ? 0 : (p >= lim ? lim - 1 : p);
}
__device__ __forceinline__ int eff_tok(const StepParams &P, int b) {
    const int t = raw_tok(P, b);
    return (t < 0 || t >= P.V) ? 0 : t;
}
__device__ __forceinline__ bool seq_ok(const StepParams &P, int b) {
    const int t = raw_tok(P, b), p = raw_pos(P, b);
    return t >= 0 && t < P.V && p >= 0 && p < min(P.cap, P.max_seq);
}
// On the per-sequence path (at most kMfmaBatch - 1 sequences) both are read once per launch
// into LDS (bar_init), so that no phase starts with a dependent memory round
// trip for them.
__device__ __forceinline__ int *seq_table(const StepParams &P);
template <bool PS>
__device__ __forceinline__ int pos_of(const StepParams &P, int b) {
    if constexpr (PS) return seq_table(P)[b];
    else return eff_pos(P, b);
}
template <bool PS>
__device__ __forceinline__ bool ok_of(const StepParams &P, int b) {
    if constexpr (PS) return seq_table(P)[kMfmaBatch + b] != 0;
    else return seq_ok(P, b);
}

__device__ __forceinline__ size_t kv_row(const StepParams &P, int l, int b, int g) {
    return (((size_t)l * P.kv_batch + b) * P.nkv + g) * (size_t)P.cap;
}

// ---------------------------------------------------------------- coherent accesses
//
// Relaxed agent-scope atomic loads and stores compile to ordinary vector
// memory instructions with the device-coherence bit (sc1): they see, and are
// seen by, every XCD without flushing or invalidating the XCD-private L2.

__device__ __forceinline__ void st_dev(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev_u16(uint16_t *p, uint16_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev_u32(unsigned *p, unsigned v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// The residual stream is kept in fixed point: int64 in units of 2^-32.  Every
// contribution (the embedding, each O-projection partial, each
// down-projection partial) is rounded once to that grid and added with an
// integer atomic, so the sum is exact and independent of the order in which
// workgroups add: results are reproducible however the work is split.  The
// range (+-2^31) and resolution (2^-32) are far beyond fp32 activations'.
constexpr double kFixScale = 4294967296.0;   // 2^32
__device__ __forceinline__ long long to_fix(float v) {
    return __double2ll_rn((double)v * kFixScale);
}
__device__ __forceinline__ float from_fix(long long v) {
    return (float)v * (1.0f / 4294967296.0f);
}
__device__ __forceinline__ void add_fix(long long *p, float v) {
    __hip_atomic_fetch_add(reinterpret_cast<unsigned long long *>(p),
                           (unsigned long long)to_fix(v), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev_u64(unsigned long long *p, unsigned long long v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float *p) {
    return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ld_dev_u64(const void *p) {
    return __hip_atomic_load(reinterpret_cast<unsigned long long *>(const_cast<void *>(p)),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ u32x4 ld_dev_16B(const void *p) {
    const unsigned long long a = ld_dev_u64(p);
    const unsigned long long b = ld_dev_u64(reinterpret_cast<const char *>(p) + 8);
    return u32x4{(unsigned)a, (unsigned)(a >> 32), (unsigned)b, (unsigned)(b >> 32)};
}
__device__ __forceinline__ u32x4 ld_stream_16B(const void *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

// Block barrier for LDS hand-offs only: the wave's LDS operations complete,
// then s_barrier; unlike __syncthreads (whose workgroup release fence also
// waits for every outstanding memory load), loads in flight stay in flight.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// s_waitcnt vmcnt(0): this wave's stores have completed at their coherence point.
__device__ __forceinline__ void wait_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// ---------------------------------------------------------------- grid barrier
//
// Arrival counting on monotonically increasing 64-bit counters, one per
// group of workgroups: workgroup w arrives on counter w % ng (one atomic
// add), and a waiter's wave 0 polls all ng counters at once, one per lane.
// Spreading arrivals over ng counters keeps the atomics on any one address
// few; polling them directly saves a second atomic hop.  The counters are
// never reset: every launch ends with counter g at E * size_g, E being the
// number of barriers completed so far, and at launch start each workgroup
// recovers E from its own group's counter.  Barrier k of a launch is complete
// when counter g reaches base_g + (k + 1) * size_g for every group g.  The
// wait is bounded by a poll count: past it, KL_DEVERR_BARRIER is raised and every
// later wait returns at once, so a broken barrier ends the kernel instead of
// hanging it.
constexpr int kSpinLimit = 1 << 22;   // polls before a wait gives up (well over a second)

// The per-group bases of the current launch live in the dynamic LDS area (a
// fixed slot after everything else; see lds_layout), which every phase
// function addresses the same way.
extern __shared__ __align__(16) char kl_smem[];
__device__ __forceinline__ unsigned long long *bar_bases(const StepParams &P);

__device__ __forceinline__ int bar_groups(const StepParams &P) { return bar_group_count(P.nwg); }
__device__ __forceinline__ unsigned bar_gsize(const StepParams &P, int ng, int g) {
    return bar_group_size(P.nwg, ng, g);
}
__device__ __forceinline__ unsigned long long *bar_counter(const StepParams &P, int g) {
    return P.bar + 32 * (g + 1);   // 256 bytes apart
}

// At launch start: the barrier bases of this launch and the step's first tag
// of the tagged hand-offs, into LDS (before any wait; any wave may do it).
__device__ __forceinline__ unsigned *launch_epoch(const StepParams &P);
__device__ __forceinline__ void bar_init(const StepParams &P) {
    // Only this workgroup's own group counter is read: that group cannot
    // complete barrier 0 before this workgroup arrives, so the value rounds
    // down to the number E of whole barriers done by earlier launches.  Any
    // other group may already be one barrier further, so its base is E times
    // its size, not its current value rounded down.
    const int ng = bar_groups(P);
    const unsigned t = kl_tid();
    if (t < (unsigned)ng) {
        const int own = blockIdx.x % ng;
        const unsigned long long c = ld_dev_u64(bar_counter(P, own));
        bar_bases(P)[t] = bar_launch_base(c, P.nwg, ng, own, (int)t);
    } else if (t == 64) {
        *launch_epoch(P) = __hip_atomic_load(P.epoch_ptr, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
    } else if (t >= 96 && t < 96 + kMfmaBatch && !P.batched) {
        const int b = (int)t - 96;
        if (b < P.B) {
            seq_table(P)[b] = eff_pos(P, b);
            seq_table(P)[kMfmaBatch + b] = seq_ok(P, b) ? 1 : 0;
        }
    }
    __syncthreads();
}

// Optional timeline: the control wave of every workgroup stamps
// (s_memrealtime, 100 MHz) the end of phase i of the launch (slot 0), the
// start and end of phase i's wait for its inputs (slots 1, 2) and the moment
// its inputs are staged (slot 3: the GEMV path's first activation vector in
// LDS, the batched path's normalised activations written by the whole grid,
// an attention phase's last chunk result published).
__device__ __forceinline__ void trace_stamp(const StepParams &P, int i, int what) {
    if (P.trace && i >= 0 && i < P.trace_max)
        P.trace[((size_t)i * P.nwg + blockIdx.x) * 4 + what] = wall_clock64();
}

// The control wave (kCtlWave) does all of a workgroup's barrier traffic.  It
// never has weight or KV loads in flight, so its polls are not queued behind
// the compute waves' prefetches (a wave's loads complete in issue order).
__device__ __forceinline__ bool is_ctl_lane0() { return kl_tid() == kCtlWave * 64; }

// Every wave drains its stores (they must be visible before the signal),
// then the control wave signals.
__device__ __forceinline__ void drain_all() {
    wait_stores();
    __syncthreads();
}

// Arrival on grid barrier k after phase ti.
// (the phase's end is stamped once every wave of the workgroup is done)
__device__ __forceinline__ void bar_arrive(const StepParams &P, int k, int ti) {
    drain_all();
    if (is_ctl_lane0()) {
        trace_stamp(P, ti, 0);
        __hip_atomic_fetch_add(bar_counter(P, blockIdx.x % bar_groups(P)), 1ull,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Arrival on a local counter (one add per arriving workgroup) after phase ti.
__device__ __forceinline__ void local_arrive(const StepParams &P, unsigned *cnt, int ti) {
    drain_all();
    if (is_ctl_lane0()) {
        trace_stamp(P, ti, 0);
        __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Spin until *flag_fn() says done; gives up (raising KL_DEVERR_BARRIER) after
// kSpinLimit polls or as soon as another wait has given up.
template <class Done>
__device__ __forceinline__ void spin_until(const StepParams &P, Done &&done) {
    for (int spins = 1;; ++spins) {
        if (done()) return;
        if ((spins & 63) == 0 &&
            (__hip_atomic_load(P.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) &
             KL_DEVERR_BARRIER))
            return;
        if (spins >= kSpinLimit) {
            if ((kl_tid() & 63) == 0)
                __hip_atomic_fetch_or(P.err, KL_DEVERR_BARRIER, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
    }
}

__device__ __forceinline__ void bar_wait(const StepParams &P, int k, int ti) {
    if ((kl_tid() >> 6) == kCtlWave) {
        const int lane = kl_tid() & 63, ng = bar_groups(P);
        const bool mine = lane < ng;
        const unsigned long long target =
            mine ? bar_target(bar_bases(P)[lane], k, P.nwg, ng, lane) : 0ull;
        if (lane == 0) trace_stamp(P, ti, 1);
        spin_until(P, [&]() {
            const bool d = !mine || bar_reached(ld_dev_u64(bar_counter(P, lane)), target);
            return __all(d) != 0;
        });
        if (lane == 0) trace_stamp(P, ti, 2);
    }
    __syncthreads();
}

// Wait until a local counter (monotonic within a step; zeroed by the
// embedding phase) reaches target.
__device__ __forceinline__ void local_wait(const StepParams &P, const unsigned *cnt,
                                           unsigned target, int ti) {
    if (is_ctl_lane0()) {
        trace_stamp(P, ti, 1);
        spin_until(P, [&]() {
            return (int)(__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) -
                         target) >= 0;
        });
        trace_stamp(P, ti, 2);
    }
    __syncthreads();
}

// ---------------------------------------------------------------- tagged hand-offs
//
// On the per-sequence path, values that cross workgroups inside a layer (the
// rotated queries and the new key and value for the attention, the chunk
// results for the O projection, the SwiGLU output for the down projection)
// travel as tagged words: one 8-byte word holds the 32-bit value and the tag
// of the step and layer that wrote it, written and read as one
// device-coherent access.  A reader polls the words themselves and takes a
// value once its tag is the current one.  The writer therefore needs no
// drain of its stores and no counter, and the reader no separate wait before
// loading: a hand-off costs the time for the stores to land plus one load
// round trip, instead of store drain, counter atomic, counter poll and data
// load one after the other.  Tags are epoch + layer, each step using a fresh
// range of tags that never includes 0 (cleared memory); the epoch is read at
// launch start and advanced by the step's last phase (ll_next_epoch).
__device__ __forceinline__ unsigned ll_tag(const StepParams &P, int l) {
    return *launch_epoch(P) + (unsigned)l;
}
__device__ __forceinline__ void st_ll(unsigned long long *p, unsigned v, unsigned tag) {
    st_dev_u64(p, ll_word(v, tag));
}
__device__ __forceinline__ void st_ll_f(unsigned long long *p, float v, unsigned tag) {
    st_ll(p, __float_as_uint(v), tag);
}

// Threads tid = 0 .. nt - 1 (the caller's numbering) gather n tagged words:
// word i (address addr(i)) goes to put(i, value) once it carries 'tag'.  Each
// thread takes words tid, tid + nt, ... in rounds of W, issuing a round's
// loads together (from in-range addresses, masked when used) and reloading
// the round until every word of it is current.  A round gives up after
// kSpinLimit polls, raising KL_DEVERR_BARRIER, so a missing writer ends the
// kernel instead of hanging it.
template <int W, class Addr, class Put>
__device__ __forceinline__ void ll_gather(const StepParams &P, int n, unsigned tag, int tid,
                                          int nt, Addr &&addr, Put &&put) {
    for (int base = 0; base < n; base += W * nt) {
        unsigned long long v[W];
        for (int spins = 1;; ++spins) {
#pragma unroll
            for (int k = 0; k < W; ++k) v[k] = ld_dev_u64(addr(min(base + tid + k * nt, n - 1)));
            bool ok = true;
#pragma unroll
            for (int k = 0; k < W; ++k) ok = ok && (base + tid + k * nt >= n || ll_current(v[k], tag));
            if (ok) break;
            if ((spins & 63) == 0 &&
                (__hip_atomic_load(P.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) &
                 KL_DEVERR_BARRIER))
                break;
            if (spins >= kSpinLimit) {
                __hip_atomic_fetch_or(P.err, KL_DEVERR_BARRIER, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
        }
#pragma unroll
        for (int k = 0; k < W; ++k)
            if (base + tid + k * nt < n) put(base + tid + k * nt, ll_value(v[k]));
    }
}

// ---------------------------------------------------------------- params
//
// The step kernel is one function per (head_dim, group size), with every
// phase inlined (no calls: a call would save and restore callee-saved
// registers through scratch memory on every phase).  Each phase reads the
// step parameters from the kernel-argument segment itself, through an
// address the compiler cannot see through, so the loads stay inside the
// phase instead of being hoisted out of the layer loop, where the values of
// all phases together would exhaust the registers.
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
    unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)ka);
    unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(ka >> 32));
    asm volatile("" : "+s"(lo), "+s"(hi));
    const KL_KARG StepParams *p = (const KL_KARG StepParams *)(((KArg)hi << 32) | lo);
    return *p;
#else
    return StepParams{};   // the host pass only type-checks device code
#endif
}

// ---------------------------------------------------------------- LDS layout

// Offsets (in floats) come from the host, which sizes the allocation.

struct Lds {
    float *a;     // activation vector (max K extent); aliased by the attention area
    float *attn;  // attention scratch (same storage as a)
    float *red;   // [kWaves][kRgBatch][kTileRows] GEMV partial sums
    float *sm;    // small reductions and flags (64 floats)
    unsigned long long *bar;   // [kBarGroups] barrier bases of this launch
};

__device__ __forceinline__ Lds lds_layout(char *smem, const StepParams &P) {
    Lds s;
    float *f = reinterpret_cast<float *>(smem);
    s.a = f;
    s.attn = f;
    s.red = f + P.lds_red;
    s.sm = f + P.lds_sm;
    s.bar = reinterpret_cast<unsigned long long *>(f + P.lds_bar);
    return s;
}
// Per-sequence path: with P.multi the B sequences share each GEMV pass and
// sequence b's staged vector sits b stride floats into the activation area
// (its wave sums of squares b kSmSeq floats into sm); otherwise every
// sequence is staged at the start of the area in turn.
__device__ __forceinline__ float *seq_vec(const StepParams &P, const Lds &S, int b, int stride) {
    return S.a + (P.multi ? b * stride : 0);
}
__device__ __forceinline__ float *seq_sm(const StepParams &P, const Lds &S, int b);
// The Q/K/V phase's staged RoPE row (cos, sin) of sequence b: after the
// activation vectors.
__device__ __forceinline__ float *rope_row(const StepParams &P, const Lds &S, int b) {
    return S.a + (P.multi ? kMultiSeq * P.Hp + b * P.d : 2 * P.Hp);
}

__device__ __forceinline__ unsigned long long *bar_bases(const StepParams &P) {
    return lds_layout(kl_smem, P).bar;
}
// (after the barrier bases)
__device__ __forceinline__ unsigned *launch_epoch(const StepParams &P) {
    return reinterpret_cast<unsigned *>(lds_layout(kl_smem, P).bar + kBarGroups);
}
// (after the epoch: position and validity of each sequence, per-sequence path)
__device__ __forceinline__ int *seq_table(const StepParams &P) {
    return reinterpret_cast<int *>(lds_layout(kl_smem, P).bar + kBarGroups) + 4;
}
// (then: the head's argmax keys of up to kGemmBatch sequences)
__device__ __forceinline__ unsigned long long *amax_slots(const StepParams &P) {
    return reinterpret_cast<unsigned long long *>(seq_table(P) + 2 * kMfmaBatch);
}
// (then, mixture of experts: per sequence, its two experts and their
// weights (float bits), chosen in the gate/up phase, used by the down phase)
__device__ __forceinline__ int *route_table(const StepParams &P) {
    return reinterpret_cast<int *>(amax_slots(P) + kGemmBatch);
}

// ---------------------------------------------------------------- activations

// Control wave only: copy 'bytes' (a multiple of 16; src and dst 16-byte
// aligned) from device memory straight to LDS (global_load_lds, 16 bytes per
// lane, device-coherent: cache-policy bits sc1), then wait for the copy.  The
// control wave has no weight loads in flight, so the copy does not queue
// behind them.
constexpr int kLdsCoherent = 16;
__device__ __forceinline__ void ctl_copy_to_lds(const void *src, void *dst, int bytes) {
    const int lane = kl_tid() & 63;
    const char *s = static_cast<const char *>(src);
    char *d = static_cast<char *>(dst);
    for (int off = 0; off < bytes; off += 64 * 16) {
        if (off + lane * 16 < bytes)
            __builtin_amdgcn_global_load_lds(s + off + lane * 16, d + off, 16, 0, kLdsCoherent);
    }
}
__device__ __forceinline__ void ctl_copy_wait() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Activation staging: loads are issued in batches of kStageBatch per thread
// before any is used.
constexpr int kStageBatch = 8;
// a[i] = x[i] * rsqrt(mean(x^2) + eps) * gain[i] for i < n, 0 up to npad,
// x read from the fixed-point residual stream.  The gain is loaded in the
// same batch as x (a dependent second batch would cost a second memory round
// trip, ~2 us when HBM is saturated), and so are the ne floats of an optional
// extra vector (esrc -> edst in LDS), e.g. the RoPE row the epilogue needs.
// RMSNorm staging for the GEMV path, with the normalisation deferred: the
// weight product is linear, so W (x r g) = r (W (x g)) with the per-sequence
// scale r = 1 / sqrt(mean(x^2) + eps) applied in the epilogue (rms_scale).
// Stages a = x g (zero padding) and leaves each wave's partial sum of x^2
// in sm[wave]; the weight stream starts as soon as a is in LDS, without
// waiting for a block-wide reduction.
__device__ __forceinline__ void stage_rms_deferred(const long long *__restrict__ xf,
                                                   const float *__restrict__ gain, int n, int npad,
                                                   float *a, float *sm,
                                                   const float *esrc = nullptr,
                                                   float *edst = nullptr, int ne = 0) {
    float ss = 0.f;
    for (int i0 = kl_tid(); i0 < npad; i0 += kStageBatch * kThreads) {
        long long v[kStageBatch];
        float gv[kStageBatch];
        float ev = 0.f;
        const bool first = i0 == (int)kl_tid();
        // (every load is unconditional, from a clamped address, and masked
        // when used: a conditional device-coherent load becomes a branch that
        // waits for its load before the next one is issued)
#pragma unroll
        for (int k = 0; k < kStageBatch; ++k) {
            const int i = i0 + k * kThreads, ic = min(i, n - 1);
            const long long xv = (long long)ld_dev_u64(xf + ic);
            const float g = gain[ic];
            v[k] = i < n ? xv : 0ll;
            gv[k] = i < n ? g : 0.f;
        }
        if (first && (int)kl_tid() < ne) ev = esrc[kl_tid()];
#pragma unroll
        for (int k = 0; k < kStageBatch; ++k) {
            const int i = i0 + k * kThreads;
            const float x = from_fix(v[k]);
            ss = fmaf(x, x, ss);
            if (i < npad) a[i] = x * gv[k];
        }
        if (first && (int)kl_tid() < ne) edst[kl_tid()] = ev;
    }
    ss = wave_sum(ss);
    if ((kl_tid() & 63) == 0) sm[kl_tid() >> 6] = ss;
    lds_barrier();
}
// The same for sequences 0 .. nb - 1 (nb <= kMultiSeq) together, their loads
// issued in one batch: sequence b's residual row at xf + b xstride, its
// staged vector at a + b astride, its wave sums at sm + b kSmSeq, and the ne
// floats esrc(b) -> edst(b).  (Loads for b >= nb repeat sequence nb - 1's
// and are dropped: every load stays unconditional.)  Half the batch per
// sequence keeps the loads in flight within the registers the weight ring
// leaves.  Each sequence's sums are those stage_rms_deferred leaves for it
// alone only up to the order of the additions: the sum of a thread's terms is
// taken in the same order, so the values are the same.
constexpr int kSmSeq = kThreads / 64;   // floats between sequences' wave sums
constexpr int kStageMulti = 4;          // loads per thread and sequence per batch
struct NoExtra {   // stage_rms_multi without an extra vector
    __device__ float *operator()(int) const { return nullptr; }
};
template <class ESrc, class EDst>
__device__ __forceinline__ void stage_rms_multi(const long long *__restrict__ xf, int xstride,
                                                const float *__restrict__ gain, int n, int npad,
                                                int nb, float *a, int astride, float *sm,
                                                ESrc &&esrc, EDst &&edst, int ne) {
    float ss[kMultiSeq];
#pragma unroll
    for (int bb = 0; bb < kMultiSeq; ++bb) ss[bb] = 0.f;
    for (int i0 = kl_tid(); i0 < npad; i0 += kStageMulti * kThreads) {
        long long v[kMultiSeq][kStageMulti];
        float gv[kStageMulti], ev[kMultiSeq];
        const bool first = i0 == (int)kl_tid();
#pragma unroll
        for (int k = 0; k < kStageMulti; ++k) {
            const int i = i0 + k * kThreads, ic = min(i, n - 1);
            const float g = gain[ic];
            gv[k] = i < n ? g : 0.f;
#pragma unroll
            for (int bb = 0; bb < kMultiSeq; ++bb) {
                const long long xv =
                    (long long)ld_dev_u64(xf + (size_t)min(bb, nb - 1) * xstride + ic);
                v[bb][k] = i < n ? xv : 0ll;
            }
        }
        if (first && (int)kl_tid() < ne) {
#pragma unroll
            for (int bb = 0; bb < kMultiSeq; ++bb) ev[bb] = esrc(min(bb, nb - 1))[kl_tid()];
        }
#pragma unroll
        for (int bb = 0; bb < kMultiSeq; ++bb) {
            if (bb < nb) {
#pragma unroll
                for (int k = 0; k < kStageMulti; ++k) {
                    const int i = i0 + k * kThreads;
                    const float x = from_fix(v[bb][k]);
                    ss[bb] = fmaf(x, x, ss[bb]);
                    if (i < npad) a[bb * astride + i] = x * gv[k];
                }
                if (first && (int)kl_tid() < ne) edst(bb)[kl_tid()] = ev[bb];
            }
        }
    }
#pragma unroll
    for (int bb = 0; bb < kMultiSeq; ++bb) {
        if (bb < nb) {
            const float t = wave_sum(ss[bb]);
            if ((kl_tid() & 63) == 0) sm[bb * kSmSeq + (kl_tid() >> 6)] = t;
        }
    }
    lds_barrier();
}
// The scale r of the sequence staged last by stage_rms_deferred (the wave
// partials are added in wave order: the same value in every thread).
__device__ __forceinline__ float rms_scale(const float *sm, int n, float eps) {
    float ss = 0.f;
#pragma unroll
    for (int w = 0; w < kSmSeq; ++w) ss += sm[w];
    return 1.0f / sqrtf(ss / (float)n + eps);
}
__device__ __forceinline__ float *seq_sm(const StepParams &P, const Lds &S, int b) {
    return S.sm + (P.multi ? b * kSmSeq : 0);
}

// ---------------------------------------------------------------- GEMV engine
//
// y_b[r] = sum_k W[r][k] a_b[k] for the rows of the row groups a workgroup owns in a
// packed matrix with KT k-tiles per row group, for each sequence b.  Each
// wave takes a fixed slice of the k-tiles of every row group (split-K inside
// the workgroup), keeps U tile loads in flight, and reduces its partial dot
// products over the 8 lanes of a row with DPP.  The slices are summed in wave
// order through LDS, and epi(b, r, y_r, y_r+1) is called once per row pair.
// Row groups are processed in batches of kRgBatch.  The first loads are
// issued before wait() (the grid barrier that publishes the activations) and
// before stage(b) (which fills a with sequence b's activation vector); each
// next batch's first loads are issued before the previous batch's reduction.
constexpr int kGemvDepth = 16;   // tile loads in flight per wave (16 KiB)
// one sequence's GEMV partial sums in the reduction area (either row sharing)
constexpr int kRedStride = kWaves * kRgBatch * kTileRows;

// The ring of tile loads must stay in flight across loop iterations, the
// grid barrier and the activation staging, and the compiler only places a
// precise "wait for the oldest load" (vmcnt(U-1)) when every path issues the
// same loads.  So the ring is refilled unconditionally: once the batch's real
// tiles are exhausted, a slot is refilled from a 16-byte dummy line that all
// lanes share (one cache line per wave), and only the consumption of a slot
// is conditional.
//
// A workgroup owns the row groups first, first + stride, ... (count of
// them).  The phases use stride 1 (a contiguous block per workgroup): a
// strided assignment (stride = grid size) was measured no faster.
struct RgRange { int first, count; };
__device__ __forceinline__ RgRange own_rgs(int nrg, const StepParams &P) {
    int a, b;
    split_range(nrg, P.nwg, blockIdx.x, a, b);
    return RgRange{a, b - a};
}

// Two ways to share a row group's tiles among the waves:
//   split-K   (long rows, KT >= 2 kWaves): wave w takes the k-tiles
//             [w KT / kWaves, (w + 1) KT / kWaves) of every row group; the
//             wave partial sums are added in wave order through LDS;
//   row-split (short rows): wave w takes whole row groups w, w + kWaves, ...
//             of the batch and needs no cross-wave sum.
// Both orders are fixed by the partition alone.
// Early (the usual case): the first ring of loads is issued before wait() and
// stage(0), overlapping their latency; otherwise after stage(0), so that the
// loads stage(0) makes are not queued behind them (a wave's loads complete in
// order).  Waves from early_from on issue theirs early in either case (they
// must then take no part in stage's loads).
template <bool RowSplit, bool Early, bool Split, class Wait, class Stage, class Epi>
__device__ __forceinline__ void gemv_rows(const uint8_t *__restrict__ W, int KT, int first,
                                          int count, int stride, int B,
                                          const float *__restrict__ a, float *red,
                                          const uint8_t *dummy, Wait &&wait, Stage &&stage,
                                          Epi &&epi, int early_from = kWaves + 1) {
    constexpr int U = kGemvDepth;
    constexpr int BATCH = RowSplit ? kWaves * kRgBatch : kRgBatch;   // row groups per LDS round
    // wave-uniform values live in scalar registers, so every branch below is
    // a scalar branch
    const int wid = __builtin_amdgcn_readfirstlane(kl_tid() >> 6);
    const int lane = kl_tid() & 63;
    const int row = lane >> 3, sub = lane & 7;
    const int kt0 = RowSplit ? 0 : (wid * KT) / kWaves;
    const int nk = RowSplit ? KT : ((wid + 1) * KT) / kWaves - kt0;
    const int rstep = RowSplit ? kWaves : 1;   // a wave's next row group, in batch items
    const uint8_t *base = W + (size_t)lane * 16;
    const float *abase = a + sub * 8;
    u32x4 buf[U];
    int n = 0, ltile = 0, lk = 0, left = 0;   // batch items; next tile, its k index; tiles left

    // from a wave's last tile of one row group to its first of the next
    const int jump = (rstep * stride - 1) * KT + (KT - nk) + 1;
    // load the next tile of the batch, or the dummy line (branch-free)
    auto load_next = [&]() {
        const int t = __builtin_amdgcn_readfirstlane(ltile);
        const bool real = left > 0;
        const u32x4 v = ld_stream_16B(real ? base + (size_t)t * kTileBytes : dummy);
        const bool wrap = lk + 1 == nk;
        ltile = real ? ltile + (wrap ? jump : 1) : ltile;
        lk = real ? (wrap ? 0 : lk + 1) : lk;
        left = real ? left - 1 : left;
        return v;
    };
    auto start = [&](int ib) {   // batch of row groups ib .. ib + BATCH - 1
        const int nb = min(BATCH, count - ib);
        const int mine = RowSplit ? (nb > wid ? (nb - wid + kWaves - 1) / kWaves : 0) : nb;
        n = nk * mine;
        left = n;
        ltile = (first + (ib + (RowSplit ? wid : 0)) * stride) * KT + kt0;
        lk = 0;
#pragma unroll
        for (int s = 0; s < U; ++s) buf[s] = load_next();
    };

    // the control wave takes part in the staging and the epilogue only
    const bool compute = wid < kWaves;
    const bool has_rows = count > 0;
    // (waves from early_from on issue their first loads early too)
    const bool early = Early || (Split && wid >= early_from);
    if (early && has_rows && compute) start(0);
    wait();
    if (!has_rows) return;
    for (int b = 0; b < B; ++b) {
        for (int ib = 0; ib < count; ib += BATCH) {
            if (early) {
                if ((b > 0 || ib > 0) && compute) start(ib);
                if (ib == 0) stage(b);
            } else {
                if (ib == 0) stage(b);
                if (compute) start(ib);
            }
            const int nrg = min(BATCH, count - ib);
            int cr = RowSplit ? wid : 0, ck = 0;   // batch item of the row group in progress
            float acc = 0.f;
            // item i sits in slot i % U and is refilled with item i + U (or
            // the dummy line) right after it is consumed
            if (compute)
            for (int i0 = 0; i0 < n; i0 += U) {
#pragma unroll
                for (int s = 0; s < U; ++s) {
                    if (i0 + s < n) {
                        const u32x4 wv = buf[s];
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
                            if (sub == 0) {
                                if (RowSplit) red[cr * kTileRows + row] = t;
                                else red[(wid * kRgBatch + cr) * kTileRows + row] = t;
                            }
                            acc = 0.f;
                            ck = 0;
                            cr += rstep;
                        }
                    }
                    buf[s] = load_next();
                }
            }
            lds_barrier();
            for (int t = kl_tid(); t < nrg * (kTileRows / 2); t += kThreads) {
                const int rgi = t / (kTileRows / 2), pr = (t % (kTileRows / 2)) * 2;
                float y0 = 0.f, y1 = 0.f;
                if (RowSplit) {
                    y0 = red[rgi * kTileRows + pr];
                    y1 = red[rgi * kTileRows + pr + 1];
                } else {
                    for (int w = 0; w < kWaves; ++w) {
                        if (((w + 1) * KT) / kWaves == (w * KT) / kWaves) continue;   // empty slice
                        y0 += red[(w * kRgBatch + rgi) * kTileRows + pr];
                        y1 += red[(w * kRgBatch + rgi) * kTileRows + pr + 1];
                    }
                }
                epi(b, (first + (ib + rgi) * stride) * kTileRows + pr, y0, y1);
            }
            lds_barrier();
        }
    }
}

// Several sequences per pass (B <= kMultiSeq): every tile is applied to all
// B staged vectors (astride floats apart; their partial sums kRedStride
// floats apart in red), so the weights stream once for all of them.  The
// activation reads from LDS then bound the pass, so a wave takes its row
// groups kMultiRg at a time, interleaved tile by tile at each k (tiles
// (r, k), (r + 1, k), ..., (r, k + 1), ...): one read of the B vectors at k
// serves kMultiRg tiles.  A group short of kMultiRg real row groups is padded
// with spare loads of the dummy line, whose products are dropped.  Every row
// group's sums are taken in the same order as in gemv_rows, so the results
// are those of B passes of one sequence.  With U a multiple of kMultiRg, a
// group's tiles sit in consecutive ring slots, known at compile time in the
// unrolled loop.
constexpr int kMultiRg = 4;
template <bool RowSplit, bool Early, bool Split, class Wait, class Stage, class Epi>
__device__ __forceinline__ void gemv_rows_multi(const uint8_t *__restrict__ W, int KT, int first,
                                                int count, int stride, int B,
                                                const float *__restrict__ a, int astride,
                                                float *red, const uint8_t *dummy, Wait &&wait,
                                                Stage &&stage, Epi &&epi, int early_from) {
    constexpr int U = kGemvDepth, NP = kMultiRg;
    static_assert(U % NP == 0, "a ring slot's place in its group must be fixed");
    constexpr int BATCH = RowSplit ? kWaves * kRgBatch : kRgBatch;
    const int wid = __builtin_amdgcn_readfirstlane(kl_tid() >> 6);
    const int lane = kl_tid() & 63;
    const int row = lane >> 3, sub = lane & 7;
    const int kt0 = RowSplit ? 0 : (wid * KT) / kWaves;
    const int nk = RowSplit ? KT : ((wid + 1) * KT) / kWaves - kt0;
    const int rsz = (RowSplit ? kWaves : 1) * stride * KT;   // tiles between a wave's row groups
    const uint8_t *base = W + (size_t)lane * 16;
    const float *abase = a + sub * 8;
    u32x4 buf[U];
    // loads: the wave's row groups gi .. gi + NP - 1 of the batch (mine of
    // them), at k index lk; tile0 = the first row group's first tile
    int n = 0, mine = 0, tile0 = 0, gi = 0, lk = 0;
    auto load_h = [&](int h) {
        const bool real = gi + h < mine;
        const int t = __builtin_amdgcn_readfirstlane(tile0 + (gi + h) * rsz + lk);
        const u32x4 v = ld_stream_16B(real ? base + (size_t)t * kTileBytes : dummy);
        if (h == NP - 1) {
            const bool wrap = lk + 1 == nk;
            lk = wrap ? 0 : lk + 1;
            gi = wrap ? gi + NP : gi;
        }
        return v;
    };
    auto start = [&](int ib) {
        const int nb = min(BATCH, count - ib);
        mine = RowSplit ? (nb > wid ? (nb - wid + kWaves - 1) / kWaves : 0) : nb;
        n = nk * NP * ((mine + NP - 1) / NP);
        tile0 = (first + (ib + (RowSplit ? wid : 0)) * stride) * KT + kt0;
        gi = 0;
        lk = 0;
#pragma unroll
        for (int s = 0; s < U; ++s) buf[s] = load_h(s % NP);
    };
    const bool compute = wid < kWaves;
    const bool has_rows = count > 0;
    const bool early = Early || (Split && wid >= early_from);
    if (early && has_rows && compute) start(0);
    wait();
    if (!has_rows) return;
    for (int ib = 0; ib < count; ib += BATCH) {
        if (early) {
            if (ib > 0 && compute) start(ib);
            if (ib == 0)
                for (int bb = 0; bb < B; ++bb) stage(bb);
        } else {
            if (ib == 0)
                for (int bb = 0; bb < B; ++bb) stage(bb);
            if (compute) start(ib);
        }
        const int nrg = min(BATCH, count - ib);
        int cr = 0, ck = 0;   // the group in progress (its first row group), its k index
        float acc[NP][kMultiSeq];
#pragma unroll
        for (int h = 0; h < NP; ++h)
#pragma unroll
            for (int bb = 0; bb < kMultiSeq; ++bb) acc[h][bb] = 0.f;
        // a group's NP tiles sit in slots s .. s + NP - 1; they are consumed
        // together (each sequence's vector read once for all of them), then
        // refilled in order
        if (compute)
        for (int i0 = 0; i0 < n; i0 += U) {
#pragma unroll
            for (int s = 0; s < U; s += NP) {
                if (i0 + s < n) {
                    float wf[NP][8];
#pragma unroll
                    for (int h = 0; h < NP; ++h) {
                        const u32x4 wv = buf[s + h];
                        wf[h][0] = bf_lo(wv.x); wf[h][1] = bf_hi(wv.x);
                        wf[h][2] = bf_lo(wv.y); wf[h][3] = bf_hi(wv.y);
                        wf[h][4] = bf_lo(wv.z); wf[h][5] = bf_hi(wv.z);
                        wf[h][6] = bf_lo(wv.w); wf[h][7] = bf_hi(wv.w);
                    }
#pragma unroll
                    for (int bb = 0; bb < kMultiSeq; ++bb) {
                        if (bb < B) {
                            const float *ap = abase + bb * astride + (kt0 + ck) * kTileK;
                            const float4 a0 = *reinterpret_cast<const float4 *>(ap);
                            const float4 a1 = *reinterpret_cast<const float4 *>(ap + 4);
                            const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
                            for (int h = 0; h < NP; ++h) {
                                float v = acc[h][bb];
#pragma unroll
                                for (int e = 0; e < 8; ++e) v = fmaf(wf[h][e], av[e], v);
                                acc[h][bb] = v;
                            }
                        }
                    }
                    if (++ck == nk) {   // the group's row groups are done
#pragma unroll
                        for (int hh = 0; hh < NP; ++hh) {
                            const int c = cr + hh;   // the wave's c-th row group of the batch
                            const int ri = RowSplit ? (wid + c * kWaves) * kTileRows + row
                                                    : (wid * kRgBatch + c) * kTileRows + row;
#pragma unroll
                            for (int bb = 0; bb < kMultiSeq; ++bb) {
                                if (bb < B) {
                                    const float t = sum8(acc[hh][bb]);
                                    if (c < mine && sub == 0) red[bb * kRedStride + ri] = t;
                                }
                                acc[hh][bb] = 0.f;
                            }
                        }
                        ck = 0;
                        cr += NP;
                    }
                }
#pragma unroll
                for (int h = 0; h < NP; ++h) buf[s + h] = load_h(h);
            }
        }
        lds_barrier();
        for (int t = kl_tid(); t < B * nrg * (kTileRows / 2); t += kThreads) {
            const int bb = t / (nrg * (kTileRows / 2)), tt = t - bb * (nrg * (kTileRows / 2));
            const int rgi = tt / (kTileRows / 2), pr = (tt % (kTileRows / 2)) * 2;
            const float *rd = red + bb * kRedStride;
            float y0 = 0.f, y1 = 0.f;
            if (RowSplit) {
                y0 = rd[rgi * kTileRows + pr];
                y1 = rd[rgi * kTileRows + pr + 1];
            } else {
                for (int w = 0; w < kWaves; ++w) {
                    if (((w + 1) * KT) / kWaves == (w * KT) / kWaves) continue;   // empty slice
                    y0 += rd[(w * kRgBatch + rgi) * kTileRows + pr];
                    y1 += rd[(w * kRgBatch + rgi) * kTileRows + pr + 1];
                }
            }
            epi(bb, (first + (ib + rgi) * stride) * kTileRows + pr, y0, y1);
        }
        lds_barrier();
    }
}

// Row groups are shared split-K when they are long enough for every wave to
// hold two or more tiles, else row-split.  Multi: the B sequences share each
// pass (gemv_rows_multi).
template <bool Early, bool Split = false, bool Multi = false, class Wait, class Stage, class Epi>
__device__ __forceinline__ void gemv_phase(const uint8_t *__restrict__ W, int KT, int first,
                                           int count, int stride, int B,
                                           const float *__restrict__ a, float *red,
                                           const uint8_t *dummy, Wait &&wait, Stage &&stage,
                                           Epi &&epi, int early_from = kWaves + 1,
                                           int astride = 0) {
    if constexpr (Multi) {
        if (KT >= 2 * kWaves)
            gemv_rows_multi<false, Early, Split>(W, KT, first, count, stride, B, a, astride, red,
                                                 dummy, wait, stage, epi, early_from);
        else
            gemv_rows_multi<true, Early, Split>(W, KT, first, count, stride, B, a, astride, red,
                                                dummy, wait, stage, epi, early_from);
    } else if (KT >= 2 * kWaves) {
        gemv_rows<false, Early, Split>(W, KT, first, count, stride, B, a, red, dummy, wait, stage,
                                       epi, early_from);
    } else {
        gemv_rows<true, Early, Split>(W, KT, first, count, stride, B, a, red, dummy, wait, stage,
                                      epi, early_from);
    }
}

// ---------------------------------------------------------------- batched engine
//
// Y[r][b] = sum_k W[r][k] X[b][k] on the matrix cores (v_mfma_f32_16x16x32_bf16:
// D[16x16] += A[16x32] B[32x16]) for the row groups first .. first + count - 1
// and up to kGemmBatch sequences b0 .. b0 + nb - 1.  A block is 16 weight
// rows (2 row groups); A = W[16 rows][32 k], B = X[32 k][16 sequences], two
// products per 32 columns cover 32 sequences, each product taken for both
// bf16 terms of X (hi, then lo, into the same accumulators).  Operand layouts:
// A lane l holds A[l % 16][8 (l / 16) .. +7], B lane l holds
// B[8 (l / 16) .. +7][l % 16], D lane l holds D[4 (l / 16) + v][l % 16].
// Weight tiles arrive through the same kind of ring of 16-byte loads as the
// GEMV path and are re-laid out through a per-wave LDS slot (2 KiB: the two
// tiles of a block at one k-tile; the slots follow the two activation chunk
// buffers).  X is staged in LDS in chunks of kGemmChunkK columns (kActStride
// bf16 per row; the hi rows, then kLoOff elements further the lo rows), in
// two chunk buffers: stage(c, buf) fills chunk c.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kLoOff = kGemmBatch * kActStride;   // elements from a chunk's hi rows to its lo rows

struct GemmLds {
    uint16_t *act[2];   // [2 terms][kGemmBatch][kActStride] bf16
};

__device__ __forceinline__ GemmLds gemm_lds(char *smem) {
    GemmLds g;
    g.act[0] = reinterpret_cast<uint16_t *>(smem);
    g.act[1] = reinterpret_cast<uint16_t *>(smem + 2 * kGemmActBytes);
    return g;
}

//
// A workgroup's products cover the row groups first .. first + count - 1 and
// the K range of W (KT k-tiles).  The K range may span several packed
// matrices of ktg k-tiles each, gstride tiles apart: k-tile kt of row group
// r is tile (kt / ktg) gstride + r ktg + kt % ktg.
//
// Work split: wave w owns the 16-row blocks w, w + kWaves, ... and takes
// them in groups of up to kGemmMaxBlk; for each group it runs through the
// chunks of K, and within a chunk through its blocks, one ring pass (U = 16
// tile loads: the 8 k-tiles of the chunk x the block's 2 row groups) per
// block.  Slot s of a pass is always (k-tile s / 2, row group s % 2), so
// that the consuming code is the same straight-line code for every pass; the
// loads run ahead through the same sequence across blocks, chunks and
// groups, and every slot is refilled unconditionally (with the zero tile
// once the wave's work is exhausted, or for a row group or k-tile past the
// range), so the compiler keeps the whole ring in flight.
//
// Activations: with up to two chunks (1024 columns) the whole K range is
// staged once and stays resident, and the waves then run without any
// workgroup barrier; longer K ranges stream through the two chunk buffers
// (the control wave copies chunk f + 1 while the compute waves work on chunk
// f; one barrier per chunk, every wave taking part in every chunk's
// barrier).  stage(c, buf) fills chunk c with the control wave's
// memory-to-LDS copies (a no-op in the other waves).
//
// Each block's products go straight from the accumulators to epi(b, r,
// y_r, y_r+1), for its row pairs and sequences b < nb.
//
// pre() runs once, after the first ring of weight loads is issued (so the
// weight stream overlaps whatever pre() waits for), before anything touches
// the activation buffers; it runs even when there are no rows.
//
// Memory-to-LDS copies issued inside the compute loop would make the
// compiler wait for all outstanding loads before each of the loop's LDS
// accesses (draining the ring once per pass), so the two modes are separate
// instances and the streaming copies run in a loop of the control wave's own.
template <bool resident, class Pre, class Stage, class Epi>
__device__ __forceinline__ void gemm_rows_mode(const uint8_t *__restrict__ W, int KT, int first,
                                               int count, int ktg, size_t gstride, int b0,
                                               int nb, const uint8_t *dummy, const GemmLds &L,
                                               Pre &&pre, Stage &&stage, Epi &&epi) {
    constexpr int U = kGemvDepth;
    constexpr int CT = kGemmChunkK / kTileK;   // k-tiles per chunk
    constexpr int MB = kGemmMaxBlk;
    static_assert(U == 2 * CT, "a ring pass is one chunk of one 16-row block");
    const int wid = __builtin_amdgcn_readfirstlane(kl_tid() >> 6);
    const int lane = kl_tid() & 63;
    const bool compute = wid < kWaves;
    const int nkc = resident ? min((KT + CT - 1) / CT, 2) : (KT + CT - 1) / CT;
    const int nblk = (count + 1) / 2;
    const int mine = (compute && nblk > wid) ? (nblk - wid + kWaves - 1) / kWaves : 0;
    const int ngrp = (mine + MB - 1) / MB;
    const int ngrp_wg = ((nblk + kWaves - 1) / kWaves + MB - 1) / MB;   // wave 0's
    const int last_rg = first + count;
    // (LDS addresses are formed from the shared array itself: a pointer taken
    // out of GemmLds by a run-time index is a generic pointer, and generic
    // loads would make every wait for an operand a wait for the whole ring)
    uint8_t *ws = reinterpret_cast<uint8_t *>(kl_smem + 4 * kGemmActBytes + wid * 2048);
    const int lo16 = lane * 16;

    // load generator: group gi, chunk gc, block gb of the group, slot gs;
    // (kg, kr) = (k-tile / ktg, k-tile % ktg) of the next load, and (kg0,
    // kr0) of the current chunk's first k-tile (wave-uniform scalars,
    // advanced by selects)
    int gi = 0, gc = 0, gb = 0, gs = 0, kg = 0, kr = 0, kg0 = 0, kr0 = 0;
    auto load_next = [&]() {
        const int blk = wid + kWaves * (MB * gi + gb);
        const int rg = first + 2 * blk + (gs & 1);
        const int kt = gc * CT + (gs >> 1);
        const bool inb = gi < ngrp && rg < last_rg && kt < KT;
        const size_t tile = (size_t)kg * gstride + (size_t)rg * ktg + kr;
        const uint8_t *src = inb ? W + tile * kTileBytes : dummy;
        const u32x4 v = ld_stream_16B(src + lo16);
        int nkr = kr + (gs & 1), nkg = kg;
        nkg = nkr == ktg ? nkg + 1 : nkg;
        nkr = nkr == ktg ? 0 : nkr;
        const bool pass_end = gs == U - 1;
        const bool blk_next = pass_end && gb + 1 < min(MB, mine - MB * gi);
        const bool chunk_end = pass_end && !blk_next;
        const bool grp_end = chunk_end && gc + 1 >= nkc;
        gs = pass_end ? 0 : gs + 1;
        gb = blk_next ? gb + 1 : (chunk_end ? 0 : gb);
        gc = grp_end ? 0 : (chunk_end ? gc + 1 : gc);
        gi = grp_end ? gi + 1 : gi;
        kg = grp_end ? 0 : (blk_next ? kg0 : nkg);
        kr = grp_end ? 0 : (blk_next ? kr0 : nkr);
        kg0 = grp_end ? 0 : (chunk_end ? nkg : kg0);
        kr0 = grp_end ? 0 : (chunk_end ? nkr : kr0);
        return v;
    };

    // (padding sequences: their rows of the activation buffers hold copies of
    // finite values; a product's columns are independent, and the outputs of
    // padding sequences are never stored)
    u32x4 buf[U];
    if (compute) {   // (the control wave keeps its load queue empty)
#pragma unroll
        for (int s = 0; s < U; ++s) buf[s] = load_next();
    }
    pre();
    if (count <= 0) return;
    __syncthreads();   // (the buffers may still hold the previous sequence group)
    stage(0, L.act[0]);
    if (resident && nkc > 1) stage(1, L.act[1]);
    __syncthreads();

    if constexpr (!resident) {
        if (!compute) {
            // chunk f + 1 into buffer (f + 1) % 2 while the compute waves work on chunk f
            const int total = ngrp_wg * nkc;
            for (int f = 0; f < total; ++f) {
                if (f + 1 < total) stage((f + 1) % nkc, L.act[(f + 1) & 1]);
                __syncthreads();
            }
            return;
        }
    }
    f32x4 acc[MB][2];
#pragma unroll
    for (int i = 0; i < MB; ++i) acc[i][0] = acc[i][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int ngl = resident ? ngrp : ngrp_wg;
    int f = 0;   // chunks consumed (streaming: chunk f sits in buffer f % 2)
    for (int g = 0; g < ngl; ++g) {
        const int nbg = min(MB, mine - MB * g);
        for (int c = 0; c < nkc; ++c, ++f) {
            const uint16_t *act = reinterpret_cast<const uint16_t *>(
                kl_smem + ((resident ? c : f) & 1) * (2 * kGemmActBytes));
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                if (i >= nbg) continue;   // (uniform)
#pragma unroll
                for (int s = 0; s < U; ++s) {
                    // tile (s % 2) of the block -> the wave's slot; the 16-byte
                    // column c of row r of tile t sits at column c ^ ((r + t) & 7),
                    // so that both these writes and the operand reads below (16
                    // rows at a time) are free of LDS bank conflicts
                    {
                        const int wr = lane >> 3, wc = lane & 7, tt = s & 1;
                        *reinterpret_cast<u32x4 *>(
                            ws + tt * 1024 + (wr * 8 + (wc ^ ((wr + tt) & 7))) * 16) = buf[s];
                    }
                    if (s & 1) {
                        const int ktl = s >> 1;
#pragma unroll
                        for (int st = 0; st < 2; ++st) {
                            const int r16 = lane & 15, ko = 4 * st + (lane >> 4);
                            const int at = r16 >> 3, ar = r16 & 7;
                            const bf16x8 a = *reinterpret_cast<const bf16x8 *>(
                                ws + at * 1024 + (ar * 8 + (ko ^ ((ar + at) & 7))) * 16);
#pragma unroll
                            for (int h = 0; h < 2; ++h) {
                                const int b = h * 16 + (lane & 15);
                                const int k = ktl * kTileK + 32 * st + 8 * (lane >> 4);
                                const bf16x8 x = *reinterpret_cast<const bf16x8 *>(
                                    act + b * kActStride + k);
                                const bf16x8 xl = *reinterpret_cast<const bf16x8 *>(
                                    act + kLoOff + b * kActStride + k);
                                acc[i][h] =
                                    __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, x, acc[i][h], 0, 0, 0);
                                acc[i][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, xl, acc[i][h],
                                                                                   0, 0, 0);
                            }
                        }
                    }
                    buf[s] = load_next();
                }
            }
            if (!resident) __syncthreads();   // chunk f consumed by every wave; f + 1 staged
        }
        // the group's products: lane l holds rows 4 (l / 16) .. + 3 of the
        // block for sequence h 16 + l % 16
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            if (i >= nbg) continue;   // (uniform)
            const int blk = wid + kWaves * (MB * g + i);
            const int r4 = 4 * (lane >> 4);
            const bool rv = first + 2 * blk + (r4 >> 3) < last_rg;
            const int r = (first + 2 * blk) * kTileRows + r4;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int b = h * 16 + (lane & 15);
                if (rv && b < nb) {
                    epi(b0 + b, r, acc[i][h][0], acc[i][h][1]);
                    epi(b0 + b, r + 2, acc[i][h][2], acc[i][h][3]);
                }
                acc[i][h] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
        }
    }
}

template <class Pre, class Stage, class Epi>
__device__ __forceinline__ void gemm_rows(const uint8_t *__restrict__ W, int KT, int first,
                                          int count, int ktg, size_t gstride, int b0, int nb,
                                          const uint8_t *dummy, const GemmLds &L, Pre &&pre,
                                          Stage &&stage, Epi &&epi) {
    if (KT <= 2 * (kGemmChunkK / kTileK))
        gemm_rows_mode<true>(W, KT, first, count, ktg, gstride, b0, nb, dummy, L, pre, stage,
                             epi);
    else
        gemm_rows_mode<false>(W, KT, first, count, ktg, gstride, b0, nb, dummy, L, pre, stage,
                              epi);
}


// ---------------------------------------------------------------- phases
//
// Synchronization between the phases of a layer (l):
//   grid barrier   after embed, oproj and down: the residual stream is
//                  complete; qkv, gateup and head wait on it.
//   cnt_qkv[g]     qkv -> attn: the workgroups of KV head g compute exactly
//                  the q/k/v rows of that head, so the attention of head g
//                  waits only for them (Sg arrivals per layer).
//   cnt_attn[g]    attn -> oproj: the chunk results of KV head g (B * C per
//                  layer), then (GEMV path, up to 4 query heads per KV head)
//                  one more arrival once the workgroup that delivered the
//                  last of them has merged them;
//                  head g's workgroups then apply the O-projection columns of
//                  head g to the merged output, adding into the residual.
//   cnt_gu[j]      gateup -> down: column block j of the FFN (Rc workgroups
//                  compute its SwiGLU values; the same Rc workgroups then
//                  apply the matching columns of the down projection).
// Local counters grow monotonically within a step (zeroed by the embedding
// phase); their targets are (l + 1) times the arrivals per layer.
// Every workgroup arrives on, and waits on, every grid barrier.

// ---------------------------------------------------------------- batched phases
//
// A weight phase runs the GEMV engine on the per-sequence path and the
// matrix-core engine otherwise (sequences in groups of kGemmBatch; the
// weights stream once per group).  In the batched path every input is staged
// as bf16 chunks: prep() runs once after wait(), both once the first weight
// loads are in flight; stageb(c, b0, nb, buf) fills chunk c for sequences
// b0 .. b0 + nb - 1 (the control wave's memory-to-LDS copies).
// (done(b0, nb) runs in every thread after the matrix-core path's group of
// sequences b0 .. b0 + nb - 1)
struct NoGroupDone {
    __device__ void operator()(int, int) const {}
};
// Per-sequence path: with P.multi, the sequences' vectors sit astride floats
// apart and share each pass (stage1(b) is called for every b before the
// pass; stage1(0) may stage them all).
template <bool BAT, bool Early = true, class Wait, class Prep, class Stage1, class StageB,
          class Epi, class Done = NoGroupDone>
__device__ __forceinline__ void weight_phase(const StepParams &P, const Lds &S,
                                             const uint8_t *W, int KT, int first, int count,
                                             Wait &&wait, Prep &&prep, Stage1 &&stage1,
                                             StageB &&stageb, Epi &&epi, int ktg = 0,
                                             size_t gstride = 0, Done done = Done(),
                                             int astride = 0) {
    if constexpr (!BAT) {
        if (P.multi)
            gemv_phase<Early, false, true>(W, KT, first, count, 1, P.B, S.a, S.red, P.dummy, wait,
                                           stage1, epi, kWaves + 1, astride);
        else
            gemv_phase<Early>(W, KT, first, count, 1, P.B, S.a, S.red, P.dummy, wait, stage1,
                              epi);
        return;
    }
    const GemmLds L = gemm_lds(kl_smem);
    for (int b0 = 0; b0 < P.B; b0 += kGemmBatch) {
        const int nb = min(kGemmBatch, P.B - b0);
        gemm_rows(W, KT, first, count, ktg ? ktg : KT, gstride, b0, nb, P.dummy, L,
                  [&]() {   // (first group only: the inputs' wait and the grid-wide prologue)
                      if (b0 == 0) {
                          wait();
                          prep();
                      }
                  },
                  [&](int c, uint16_t *buf) { stageb(c, b0, nb, buf); }, epi);
        done(b0, nb);
    }
}

// Batched RMSNorm (Sec. 2), deferred scale.  The K-slice partial sums of
// the last O or down projection (nparts of them) are first folded into the
// residual, x = x_in + sum_s fix(part_s) (exact integer adds, so the order is
// immaterial), and x is written to x_out; act / act_lo = the two bf16 terms
// of x gain, and the row's sum of squares goes to P.ssp per kGemmChunkK
// columns.  The consumers apply r = 1 / rms(x) to the products (rms_r).
// Items (sequence, kGemmChunkK-column slice) are spread over the grid, one
// column per thread.  Each item arrives on its slice's counter (norm_cnt,
// B arrivals per slice per RMSNorm step); a product waits only for the
// slices it stages (norm_wait) instead of on a grid barrier.  The counters
// sit kNormCntStride words apart: on one shared line, the polls of every
// control wave and the items' atomics contend (measured slower than the
// grid barrier).
__device__ __forceinline__ unsigned *norm_cnt(const StepParams &P) {
    return P.cnt + 2 * P.nkv + P.Sc;
}
__device__ __forceinline__ void norm_batched(const StepParams &P, const Lds &S,
                                             const float *gain, const long long *xin,
                                             long long *xout, int nparts) {
    static_assert(kGemmChunkK <= kThreads, "one column per thread");
    const int ns = (P.Hp + kGemmChunkK - 1) / kGemmChunkK;
    const int plast = max(nparts - 1, 0);
    for (int it = blockIdx.x; it < P.B * ns; it += P.nwg) {
        const int b = it / ns, sl = it % ns;
        const int i = sl * kGemmChunkK + (int)kl_tid();
        const bool live = (int)kl_tid() < kGemmChunkK && i < P.Hp;
        const int ic = min(i, P.Hp - 1);
        // (unconditional loads from in-range addresses, masked when used)
        long long x = (long long)ld_dev_u64(xin + (size_t)b * P.Hp + ic);
        const float *pr = P.xpart + (size_t)b * P.Hp + ic;
        float pv[kMaxKSlices];
#pragma unroll
        for (int q = 0; q < kMaxKSlices; ++q)
            pv[q] = ld_dev(pr + (size_t)min(q, plast) * P.xpart_stride);
#pragma unroll
        for (int q = 0; q < kMaxKSlices; ++q)
            if (q < nparts) x += to_fix(pv[q]);
        float ss = 0.f;
        if (live) {
            const float xv = from_fix(x);
            ss = xv * xv;   // (padding columns hold zero)
            if (nparts > 0)
                st_dev_u64(reinterpret_cast<unsigned long long *>(xout + (size_t)b * P.Hp + i),
                           (unsigned long long)x);
            uint16_t hi, lo;
            split_bf16(xv * gain[i], hi, lo);
            st_dev_u16(P.act + (size_t)b * P.Hp + i, hi);
            st_dev_u16(P.act_lo + (size_t)b * P.Hp + i, lo);
        }
        ss = block_sum(ss, S.sm);
        if (kl_tid() == 0) st_dev(P.ssp + (size_t)b * ns + sl, ss);
        drain_all();   // (also: S.sm is reused by the next item)
        if (is_ctl_lane0())
            __hip_atomic_fetch_add(norm_cnt(P) + kNormCntStride * sl, 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    }
}

// The control wave waits until the slices [c0, c1) of RMSNorm step inst
// (numbered within the step: 2 l for layer l's attention norm, 2 l + 1 for
// its FFN norm, 2 L for the final norm) are complete.  No workgroup barrier:
// the control wave then copies those slices (the other waves meet it at the
// barrier after the copies).
__device__ __forceinline__ void norm_wait(const StepParams &P, int inst, int c0, int c1) {
    if (is_ctl_lane0()) {
        const unsigned target = (unsigned)(inst + 1) * (unsigned)P.B;
        for (int c = c0; c < c1; ++c)
            spin_until(P, [&]() {
                return (int)(__hip_atomic_load(norm_cnt(P) + kNormCntStride * c, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT) - target) >= 0;
            });
    }
}

// (the steps that apply the scales keep those of sequences below
// kRScaleTable in LDS, in the area of the GEMV partial sums, which the
// batched path does not use)
constexpr int kRScaleTable = kWaves * kRgBatch * kTileRows;

// 1 / rms of sequence b's row normalised by the last batched RMSNorm step
// (its column-slice sums of squares, added in slice order).
__device__ __forceinline__ float rms_r(const StepParams &P, int b) {
    const int ns = (P.Hp + kGemmChunkK - 1) / kGemmChunkK;
    float ss = 0.f;
    for (int s0 = 0; s0 < ns; s0 += 16) {
        float v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = ld_dev(P.ssp + (size_t)b * ns + min(s0 + j, ns - 1));
#pragma unroll
        for (int j = 0; j < 16; ++j)
            if (s0 + j < ns) ss += v[j];
    }
    return 1.0f / sqrtf(ss / (float)P.H + P.eps);
}

// The scales rms_r of sequences below kRScaleTable, in LDS (S.red), for
// the steps that fold a batched product's partials; ends with a workgroup
// barrier.
__device__ __forceinline__ void rms_table(const StepParams &P, const Lds &S) {
    for (int t = kl_tid(); t < min(P.B, kRScaleTable); t += kThreads) S.red[t] = rms_r(P, t);
    __syncthreads();
}
__device__ __forceinline__ float rms_of(const StepParams &P, const Lds &S, int b) {
    return b < kRScaleTable ? S.red[b] : rms_r(P, b);
}

// Chunk c of the normalised activations (control wave: memory-to-LDS copies).
//
// Rows k0 .. k0 + kc - 1 (kc <= kGemmChunkK: one 16-byte copy per lane and row)
// of both terms of sequences b0 .. b0 + nb - 1 of a two-term bf16 matrix with
// row stride ld.  The copies are straight-line code without branches: a
// branch or loop between two copies makes the compiler wait for the first
// before issuing the second (it cannot tell that their LDS ranges are
// disjoint).  So every padding row (b >= nb) receives a copy of row nb - 1,
// and lanes past kc copy a clamped in-row address: the matrix-core loop
// reads neither (outputs of padding sequences are discarded, columns past
// kc are never consumed).
__device__ __forceinline__ void ctl_copy_rows(const uint16_t *hi, const uint16_t *lo, int ld,
                                              int k0, int kc, int b0, int nb, uint16_t *buf) {
    if ((kl_tid() >> 6) != kCtlWave) return;
    const int lane = kl_tid() & 63;
    const uint64_t col = (uint64_t)(k0 + min(lane * 8, kc - 8));
    // (the row offset is opaque to the compiler at each step, so that the
    // addresses are formed right before their copies instead of all at once)
    uint64_t row = (uint64_t)b0 * ld;
    const uint64_t last = (uint64_t)(b0 + nb - 1) * ld;
#pragma unroll
    for (int b = 0; b < kGemmBatch; ++b) {
        const uint64_t o = min(row, last) + col;
        __builtin_amdgcn_global_load_lds(hi + o, buf + b * kActStride, 16, 0, kLdsCoherent);
        __builtin_amdgcn_global_load_lds(lo + o, buf + kLoOff + b * kActStride, 16, 0,
                                         kLdsCoherent);
        row += (uint64_t)ld;
        asm volatile("" : "+v"(row));
    }
    ctl_copy_wait();
}

__device__ __forceinline__ void stage_act_chunk(const StepParams &P, int c, int b0, int nb,
                                                uint16_t *buf) {
    const int k0 = c * kGemmChunkK;
    ctl_copy_rows(P.act, P.act_lo, P.Hp, k0, min(kGemmChunkK, P.Hp - k0), b0, nb, buf);
}

// Chunk c of a two-term bf16 matrix src / src_lo [b][ld] with K columns
// (control wave: memory-to-LDS copies, so the compute waves keep working on
// the previous chunk).
__device__ __forceinline__ void stage_bf16_chunk(const uint16_t *src, const uint16_t *src_lo,
                                                 int ld, int K, int c, int b0, int nb,
                                                 uint16_t *buf) {
    const int k0 = c * kGemmChunkK;
    ctl_copy_rows(src, src_lo, ld, k0, min(kGemmChunkK, K - k0), b0, nb, buf);
}

// Batched path, several attention chunks per (sequence, KV head): the merged
// attention output o_h = sum_c w_ch A_ch / sum_c w_ch L_ch, w_ch =
// exp(M_ch - M_h) (Sec. 2 attention, split over the context), as the two
// bf16 terms the O projection stages; elements spread over the grid.  Ends
// with grid barrier k.
template <int D, int G>
__device__ __forceinline__ void merge_batched(const StepParams &P, int k) {
    const int C = P.C, n = P.nq * D, total = P.B * n;
    for (int e = blockIdx.x * kThreads + kl_tid(); e < total; e += P.nwg * kThreads) {
        const int b = e / n, j = e % n, h = j / D, g = h / G, hl = h % G, dd = j % D;
        const size_t item0 = ((size_t)b * P.nkv + g) * C;
        float M = -INFINITY;
        for (int cc = 0; cc < C; ++cc)
            M = fmaxf(M, ld_dev(P.part_s + ((item0 + cc) * G + hl) * 2));
        float num = 0.f, den = 0.f;
        for (int cc = 0; cc < C; ++cc) {
            const float m = ld_dev(P.part_s + ((item0 + cc) * G + hl) * 2);
            const float w = (m == -INFINITY) ? 0.f : expf(m - M);
            num = fmaf(ld_dev(P.part_o + (item0 + cc) * G * D + hl * D + dd), w, num);
            den = fmaf(ld_dev(P.part_s + ((item0 + cc) * G + hl) * 2 + 1), w, den);
        }
        uint16_t hi, lo;
        split_bf16(num / den, hi, lo);
        st_dev_u16(P.acto + (size_t)b * n + j, hi);
        st_dev_u16(P.acto_lo + (size_t)b * n + j, lo);
    }
    bar_arrive(P, k, -1);
    bar_wait(P, k, -1);
}

// Embedding block (Sec. 2): x = E[token] (exact in fixed point).  Workgroup 0
// records bad token ids and positions, and zeroes the local counters.
__device__ __forceinline__ void phase_embed(KArg ka, int gwait, int garrive, int ti) {
    const StepParams P = load_params(ka);
    if (gwait >= 0) bar_wait(P, gwait, ti);
    if (blockIdx.x == 0) {
        for (int b = kl_tid(); b < P.B; b += kThreads) {
            const int t = raw_tok(P, b), p = raw_pos(P, b);
            int bits = 0;
            if (t < 0 || t >= P.V) bits |= KL_DEVERR_TOKEN;
            if (p < 0 || p >= P.cap || p >= P.max_seq) bits |= KL_DEVERR_POSITION;
            if (bits) atomicOr(P.err, bits);
            // token loop: record the token taken, clear this step's argmax
            if (P.tok_emit) P.tok_emit[b] = t;
            if (P.amax) st_dev_u64(P.amax + b, 0ull);
        }
        // (the batched RMSNorm counters exist, and are used, in batched steps only)
        const int nc = 2 * P.nkv + P.Sc +
                       (P.batched ? kNormCntStride * ((P.Hp + kGemmChunkK - 1) / kGemmChunkK) : 0);
        for (int i = kl_tid(); i < nc; i += kThreads)
            __hip_atomic_store(P.cnt + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const int total = P.B * P.Hp;
    for (int idx = blockIdx.x * kThreads + kl_tid(); idx < total; idx += P.nwg * kThreads) {
        const int b = idx / P.Hp, i = idx % P.Hp;
        const float e = (i < P.H) ? bf2f(P.embed[(size_t)eff_tok(P, b) * P.H + i]) : 0.f;
        st_dev_u64(reinterpret_cast<unsigned long long *>(P.xf + idx),
                   (unsigned long long)to_fix(e));
    }
    if (garrive >= 0) bar_arrive(P, garrive, ti);
}

// One rotation pair (rows lr, lr + 1 of KV head g's block, lr even) of the
// q/k/v projection of sequence b: RoPE (Sec. 2) on query and key rows with
// cs = (cos, sin) of the pair's angle at the sequence's position, then the
// key and value to the KV cache at that position, and the query (and the new
// key and value, for the attention) to the attention's inputs: tagged words
// (LL, the per-sequence path, tag 'tag') or plain device-coherent stores.
template <bool LL, class Rope>
__device__ __forceinline__ void qkv_store(const StepParams &P, int l, int b, int g, int lr,
                                          float y0, float y1, Rope &&rope, unsigned tag = 0) {
    const int d = P.d, half = P.d / 2, G = P.group;
    const int p = pos_of<LL>(P, b);
    const bool ok = ok_of<LL>(P, b);
    unsigned long long *kvl = LL ? P.kv_ll + ((size_t)b * P.nkv + g) * d : nullptr;
    if (lr < (G + 1) * d) {
        const int i = (lr % d) >> 1;
        const float2 cs = rope(p, i);
        const float u0 = y0 * cs.x - y1 * cs.y;
        const float u1 = y0 * cs.y + y1 * cs.x;
        if (lr < G * d) {
            const size_t qo = (size_t)b * P.nq * d + (size_t)(g * G + lr / d) * d;
            if (LL) {
                st_ll_f(P.q_ll + qo + i, u0, tag);
                st_ll_f(P.q_ll + qo + i + half, u1, tag);
            } else {
                st_dev(P.q + qo + i, u0);
                st_dev(P.q + qo + i + half, u1);
            }
        } else {
            const uint16_t k0 = f2bf(u0), k1 = f2bf(u1);
            if (ok) {
                uint16_t *kk = P.kc + (kv_row(P, l, b, g) + p) * d;
                st_dev_u16(kk + i, k0);
                st_dev_u16(kk + i + half, k1);
            }
            if (LL) st_ll(kvl + i, (unsigned)k0 | ((unsigned)k1 << 16), tag);
        }
    } else {
        const int j = lr - (G + 1) * d;
        const unsigned v01 = (unsigned)f2bf(y0) | ((unsigned)f2bf(y1) << 16);
        if (ok) {
            uint16_t *vv = P.vc + (kv_row(P, l, b, g) + p) * d;
            st_dev_u32(reinterpret_cast<unsigned *>(vv + j), v01);
        }
        if (LL) st_ll(kvl + half + j / 2, v01, tag);
    }
}

// Batched path: KV head g's q/k/v rows from the K-slice partials (sums in
// slice order), through qkv_store, by head g's workgroups (part of Sg).
__device__ __forceinline__ void fold_qkv(const StepParams &P, const Lds &S, int l, int g,
                                         int part) {
    const int hrows = P.qkv_rg * kTileRows, rows = P.nkv * hrows, KS = P.KSq;
    rms_table(P, S);
    const int npair = hrows / 2, total = P.B * npair, half = P.d / 2;
    for (int e = part * kThreads + kl_tid(); e < total; e += P.Sg * kThreads) {
        const int b = e / npair, lr = 2 * (e % npair);
        const float *src = P.gpart + (size_t)b * rows + g * hrows + lr;
        float y0 = 0.f, y1 = 0.f;
        for (int q0 = 0; q0 < KS; q0 += 4) {
            // (unconditional loads from in-range addresses, masked when used)
            unsigned long long v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                v[j] = ld_dev_u64(src + (size_t)min(q0 + j, KS - 1) * P.qpart_stride);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (q0 + j < KS) {
                    y0 += __uint_as_float((unsigned)v[j]);
                    y1 += __uint_as_float((unsigned)(v[j] >> 32));
                }
            }
        }
        const float r = rms_of(P, S, b);   // the deferred RMSNorm scale
        y0 *= r;
        y1 *= r;
        if (P.qkv_bias) {   // (packed row order)
            const float *bias = reinterpret_cast<const float *>(
                P.arena + (size_t)l * P.layer_stride + P.off_qkv_bias);
            y0 += bias[g * hrows + lr];
            y1 += bias[g * hrows + lr + 1];
        }
        qkv_store<false>(P, l, b, g, lr, y0, y1,
                         [&](int p, int i) { return P.rope[(size_t)p * half + i]; });
    }
}

// RMSNorm + Q/K/V projection of KV head g + RoPE + KV-cache append.  The rows
// of head g's block are: its G query heads, then its key, then its value
// head; query and key rows are packed in rotation pairs (dims i, i + d/2).
// Batched path: a 2-D partition (KSq K slices x row groups of all heads)
// writes K-slice partials; after grid barrier qbar head g's workgroups fold
// them (fold_qkv).
template <bool BAT>
__device__ __forceinline__ void phase_qkv(KArg ka, int l, int gwait, int qbar, int ti) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    const int g = blockIdx.x / P.Sg, part = blockIdx.x % P.Sg;
    const bool member = g < P.nkv;
    const uint8_t *Lb = P.arena + (size_t)l * P.layer_stride;
    const float *gain = reinterpret_cast<const float *>(Lb + P.off_attn_norm);
    const int half = P.d / 2;
    if constexpr (BAT) {
        const int KS = P.KSq, RB = P.nwg / KS, KT = P.Hp / kTileK, KTs = KT / KS;
        const int ks = blockIdx.x / RB, rb = blockIdx.x % RB, ksc = min(ks, KS - 1);
        const int nrg = P.nkv * P.qkv_rg, rows = nrg * kTileRows;
        int a0 = 0, a1 = 0;
        if (ks < KS) split_range(nrg, RB, rb, a0, a1);
        const int col0 = ksc * KTs * kTileK;
        float *pp = P.gpart + (size_t)ksc * P.qpart_stride;
        weight_phase<true>(
            P, S, Lb + P.off_qkv + (size_t)ksc * KTs * kTileBytes, KTs, a0, a1 - a0,
            [&]() { if (gwait >= 0) bar_wait(P, gwait, ti); },
            // (layer 0 reads the embedding; later layers fold the down
            // projection's partials, x: xf2 -> xf)
            [&]() {
                norm_batched(P, S, gain, l == 0 ? P.xf : P.xf2, P.xf, l == 0 ? 0 : P.KSd);
                if (is_ctl_lane0()) trace_stamp(P, ti, 3);
            },
            [&](int) {},
            [&](int c, int b0, int nb, uint16_t *buf) {
                const int sl = col0 / kGemmChunkK + c;
                if (b0 == 0) norm_wait(P, 2 * l, sl, sl + 1);
                stage_bf16_chunk(P.act + col0, P.act_lo + col0, P.Hp, KTs * kTileK, c, b0, nb, buf);
            },
            [&](int b, int r, float y0, float y1) {
                st_dev(pp + (size_t)b * rows + r, y0);
                st_dev(pp + (size_t)b * rows + r + 1, y1);
            },
            KT, 0);
        bar_arrive(P, qbar, -1);
        bar_wait(P, qbar, -1);
        if (member) {
            fold_qkv(P, S, l, g, part);
            local_arrive(P, P.cnt + g, ti);
        }
        return;
    }
    int a0 = 0, a1 = 0;
    if (member) split_range(P.qkv_rg, P.Sg, part, a0, a1);
    const int row0 = g * P.qkv_rg * kTileRows;   // first packed row of head g's block
    weight_phase<false>(
        P, S, Lb + P.off_qkv, P.Hp / kTileK, g * P.qkv_rg + a0, a1 - a0,
        [&]() { if (gwait >= 0) bar_wait(P, gwait, ti); }, [&]() {},
        [&](int b) {
            // the RoPE row of the sequence's position rides along (rope_row)
            auto rsrc = [&](int bb) {
                return reinterpret_cast<const float *>(P.rope +
                                                       (size_t)pos_of<true>(P, bb) * half);
            };
            if (P.multi) {
                if (b == 0)
                    stage_rms_multi(P.xf, P.Hp, gain, P.H, P.Hp, P.B, S.a, P.Hp, S.sm, rsrc,
                                    [&](int bb) { return rope_row(P, S, bb); }, 2 * half);
            } else {
                stage_rms_deferred(P.xf + (size_t)b * P.Hp, gain, P.H, P.Hp, S.a, S.sm, rsrc(b),
                                   rope_row(P, S, b), 2 * half);
            }
            if (b == 0 && is_ctl_lane0()) trace_stamp(P, ti, 3);
        },
        [&](int, int, int, uint16_t *) {},
        [&](int b, int r, float y0, float y1) {
            // the deferred RMSNorm scale
            const float rs = rms_scale(seq_sm(P, S, b), P.H, P.eps);
            y0 *= rs;
            y1 *= rs;
            if (P.qkv_bias) {   // (packed row order)
                const float *bias = reinterpret_cast<const float *>(Lb + P.off_qkv_bias);
                y0 += bias[r];
                y1 += bias[r + 1];
            }
            qkv_store<true>(P, l, b, g, r - row0, y0, y1, [&](int, int i) {
                return reinterpret_cast<const float2 *>(rope_row(P, S, b))[i];
            }, ll_tag(P, l));
        },
        0, 0, NoGroupDone(), P.Hp);
    // (the attention polls the tagged words: no drain, no counter)
    if (is_ctl_lane0()) trace_stamp(P, ti, 0);
}

// The merged attention output of query head hq of KV head g for sequence b
// (Sec. 2 attention, split over the context): o = sum_c w_c A_c / sum_c w_c
// L_c with w_c = exp(M_c - M), M the largest chunk maximum, over the C chunk
// results (A_c the unnormalised output, M_c the maximum, L_c the sum of the
// chunk).  The results arrive as tagged words, kMergeChunks chunks per round;
// a later round rescales the running sums to its new maximum.  Chunks are
// taken in order, so the sums are the same in every schedule.  Threads
// 0 .. NT - 1 gather the results; leaves o[0 .. D) (LDS), with the LDS
// area scr for the chunk results.
template <int D, int G, int NT = kThreads>
__device__ __forceinline__ void merge_ll(const StepParams &P, int l, int b, int g, int hq,
                                         float *o, float *scr) {
    constexpr int WD = D + 2;                       // words per chunk and head
    float *wts = scr;                               // [kMergeChunks]
    float *run = wts + kMergeChunks;                // running max, running sum, rescale
    float *raw = run + 4;                           // [kMergeChunks][D + 2] values
    const unsigned tag = ll_tag(P, l);
    const int C = P.C;
    // chunk c's words of query head hq: src + c (D + 2) + j (contiguous)
    const unsigned long long *src = P.po_ll + (((size_t)b * P.nkv + g) * G + hq) * C * WD;
    auto val = [&](int i) { return raw[i]; };
    for (int c0 = 0; c0 < C; c0 += kMergeChunks) {
        const int nc = min(kMergeChunks, C - c0);
        if (NT == kThreads || kl_tid() < NT)
            ll_gather<(kMergeChunks * WD + NT - 1) / NT>(
                P, nc * WD, tag, kl_tid(), NT, [&](int i) { return src + (size_t)c0 * WD + i; },
                [&](int i, unsigned v) { raw[i] = __uint_as_float(v); });
        lds_barrier();
        if (kl_tid() < 64) {   // wave 0: this round's chunk weights and sum
            const int lane = kl_tid();
            float mx = -INFINITY;
            for (int c = lane; c < nc; c += 64) mx = fmaxf(mx, val(c * WD + D));
            mx = wave_max(mx);
            const float mold = c0 == 0 ? -INFINITY : run[0];
            const float mnew = fmaxf(mold, mx);
            float den = 0.f;
            for (int c = lane; c < nc; c += 64) {
                const float m = val(c * WD + D);
                const float w = (m == -INFINITY) ? 0.f : expf(m - mnew);
                wts[c] = w;
                den = fmaf(val(c * WD + D + 1), w, den);
            }
            den = wave_sum(den);
            if (lane == 0) {
                const float resc = (mold == -INFINITY) ? 0.f : expf(mold - mnew);
                run[1] = (c0 == 0 ? 0.f : run[1] * resc) + den;
                run[2] = resc;
                run[0] = mnew;
            }
        }
        lds_barrier();
        for (int t = kl_tid(); t < D; t += kThreads) {
            float acc = c0 == 0 ? 0.f : o[t] * run[2];
            for (int c = 0; c < nc; ++c) acc = fmaf(wts[c], val(c * WD + t), acc);
            o[t] = acc;
        }
        lds_barrier();
    }
    for (int t = kl_tid(); t < D; t += kThreads) o[t] = o[t] / run[1];
    lds_barrier();
}
// The same for sequences 0 .. nb - 1 together (nb C <= kMergeChunks): one
// gather of all their chunk results, then wave b forms sequence b's chunk
// weights and sum; sequence b's output goes to S.a + b D.  Each output is
// the one merge_ll gives for its sequence alone (a single round there).
template <int D, int G, int NT = kThreads>
__device__ __forceinline__ void merge_ll_multi(const StepParams &P, int l, int nb, int g, int hq,
                                               const Lds &S) {
    constexpr int WD = D + 2;
    float *wts = S.a + kMultiSeq * D;               // [nb][C]
    float *den = wts + kMergeChunks;                // [nb]
    float *raw = den + 4;                           // [nb][C][D + 2] values
    const unsigned tag = ll_tag(P, l);
    const int C = P.C, per = C * WD;
    const size_t sstride = (size_t)P.nkv * G * per;   // words between sequences
    const unsigned long long *src = P.po_ll + ((size_t)g * G + hq) * per;
    if (NT == kThreads || kl_tid() < NT)
        ll_gather<(kMergeChunks * WD + NT - 1) / NT>(
            P, nb * per, tag, kl_tid(), NT,
            [&](int i) {
                const int bb = i / per;
                return src + bb * sstride + (i - bb * per);
            },
            [&](int i, unsigned v) { raw[i] = __uint_as_float(v); });
    lds_barrier();
    const int wid = kl_tid() >> 6;
    if (wid < nb) {
        const int lane = kl_tid() & 63;
        const float *rv = raw + wid * per;
        float mx = -INFINITY;
        for (int c = lane; c < C; c += 64) mx = fmaxf(mx, rv[c * WD + D]);
        mx = wave_max(mx);
        float dn = 0.f;
        for (int c = lane; c < C; c += 64) {
            const float m = rv[c * WD + D];
            const float w = (m == -INFINITY) ? 0.f : expf(m - mx);
            wts[wid * C + c] = w;
            dn = fmaf(rv[c * WD + D + 1], w, dn);
        }
        dn = wave_sum(dn);
        if (lane == 0) den[wid] = 0.f + dn;
    }
    lds_barrier();
    for (int t = kl_tid(); t < nb * D; t += kThreads) {
        const int bb = t / D, j = t - bb * D;
        const float *rv = raw + bb * per;
        float acc = 0.f;
        for (int c = 0; c < C; ++c) acc = fmaf(wts[bb * C + c], rv[c * WD + j], acc);
        S.a[bb * D + j] = acc / den[bb];
    }
    lds_barrier();
}

// One attention work item of the per-sequence path with up to 4 query heads
// per KV head, where a chunk is short (at batch 1: 128 positions): chunk c of
// sequence b against KV head g, for the G query heads of that group
// (split-K flash decoding).  Positions are grouped in slabs of PP positions
// (one 16-byte load per lane covers a slab); chunk c owns a contiguous range
// of slabs, and inside a sub-chunk slab q is held by wave q % kWaves, so
// every compute wave takes part even when a chunk is short.  The scores of a
// sub-chunk go through LDS to a block softmax (wave h for head h), then the
// values.  Scores and probabilities are fp32.  The chunk's K/V vectors are
// loaded before the wait for the queries, except the new slot, which the
// Q/K/V phase hands over as tagged words with the queries; loads are
// unconditional (spare ones target a shared 16-byte line) and masked when
// consumed.  The chunk result (max, sum, unnormalised output per head)
// leaves as tagged words.  (At these chunk lengths this form measured
// faster than the streaming item below: 9.8 against 10.6 us per layer.)
template <int D, int NG>
constexpr int attn_sub() { return kWaves * NG * (64 / (D / 8)); }

template <int D, int G>
__device__ __forceinline__ void attn_item_ll(KArg ka, int l, int b, int g, int c, int ti) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    constexpr int LP = D / 8;                       // lanes per position
    constexpr int PP = 64 / LP;                     // positions per slab
    constexpr int NG = kAttnLoads;                  // slabs per wave per sub-chunk
    constexpr int SUB = attn_sub<D, NG>();          // positions per sub-chunk
    const int wid = __builtin_amdgcn_readfirstlane(kl_tid() >> 6);
    const int lane = kl_tid() & 63;
    const int pi = lane / LP, ds = (lane % LP) * 8;
    const int pnew = pos_of<true>(P, b), n = pnew + 1;
    int s0, s1;
    split_range((n + PP - 1) / PP, P.C, c, s0, s1);
    const int j0 = min(n, s0 * PP), j1 = min(n, s1 * PP);
    const bool compute = wid < kWaves;

    float *qs = S.attn;                 // [G][D]
    float *sp = qs + G * D;             // [G][SUB]
    float *st = sp + G * SUB;           // [G][4]: max, sum, rescale
    float *red = st + G * 4;            // [kWaves][G][D]
    uint16_t *kn = reinterpret_cast<uint16_t *>(red + kWaves * G * D);   // [D] new key
    uint16_t *vn = kn + D;                                               // [D] new value
    const size_t row0 = kv_row(P, l, b, g);
    const uint16_t *Kb = P.kc + row0 * D;
    const uint16_t *Vb = P.vc + row0 * D;
    const float scale = 1.0f / sqrtf((float)D);

    // local position of (wave, load t) in a sub-chunk
    auto jloc = [&](int t) { return (t * kWaves + wid) * PP + pi; };
    u32x4 kr[NG], vr[NG];
    // K (or V) vectors of a sub-chunk; the next sub-chunk's K is issued once
    // the scores have used this one's, and its V once the values have (the
    // loop is software-pipelined over sub-chunks)
    auto issue_one = [&](u32x4 *r, const uint16_t *base, int js, int len) {
#pragma unroll
        for (int t = 0; t < NG; ++t) {
            const int jl = jloc(t), pos = js + jl;
            const bool real = jl < len && pos != pnew;
            r[t] = ld_stream_16B(real ? (const void *)(base + (size_t)pos * D + ds) : P.dummy);
        }
    };
    if (compute) {   // (the control wave keeps its load queue empty for the barrier)
        issue_one(kr, Kb, j0, min(SUB, j1 - j0));
        issue_one(vr, Vb, j0, min(SUB, j1 - j0));
    }
    // the new slot (written during this step by another workgroup) arrives
    // as tagged words; the lanes that hold it take it from LDS after the wait,
    // into registers of their own, in place of their ring value (no ring
    // load is conditional, so the compiler's waits for the ring stay exact)
    u32x4 knew = {0u, 0u, 0u, 0u}, vnew = {0u, 0u, 0u, 0u};
    const int pl = (pnew - j0) % SUB;   // its place in its sub-chunk
    const bool holds_new =
        compute && pnew >= j0 && pnew < j1 && (pl / PP) % kWaves == wid && pl % PP == pi;
    {
        // the queries of head g's query heads and the new key and value, as
        // tagged words (every thread takes a few), into LDS
        if (is_ctl_lane0()) trace_stamp(P, ti, 1);
        const size_t qo = (size_t)b * P.nq * D + (size_t)g * G * D;
        const unsigned long long *kvl = P.kv_ll + ((size_t)b * P.nkv + g) * D;
        ll_gather<(G * D + D + kThreads - 1) / kThreads>(
            P, G * D + D, ll_tag(P, l), kl_tid(), kThreads,
            [&](int i) { return i < G * D ? P.q_ll + qo + i : kvl + (i - G * D); },
            [&](int i, unsigned v) {
                if (i < G * D) {
                    qs[i] = __uint_as_float(v);
                } else if (i < G * D + D / 2) {   // key dims j and j + D/2
                    const int j = i - G * D;
                    kn[j] = (uint16_t)v;
                    kn[j + D / 2] = (uint16_t)(v >> 16);
                } else {                           // value dims 2j and 2j + 1
                    reinterpret_cast<unsigned *>(vn)[i - G * D - D / 2] = v;
                }
            });
    }
    if (kl_tid() < G) {
        st[kl_tid() * 4 + 0] = -INFINITY;
        st[kl_tid() * 4 + 1] = 0.f;
    }
    lds_barrier();
    if (is_ctl_lane0()) trace_stamp(P, ti, 2);
    if (holds_new) {
        knew = *reinterpret_cast<const u32x4 *>(kn + ds);
        vnew = *reinterpret_cast<const u32x4 *>(vn + ds);
    }
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;

    // (the loop is split by role: in the compute waves' copy every ring load
    // is consumed on every path, so the compiler's waits stay exact; the
    // control wave takes part in the barriers only)
    if (!compute) {
        for (int js = j0; js < j1; js += SUB) {
            lds_barrier();
            lds_barrier();
            lds_barrier();
        }
    } else {
        // one sub-chunk; refill: issue the next sub-chunk's loads (every
        // sub-chunk but the last; decided at run time: a chunk is mostly one
        // sub-chunk here, where a peeled last copy costs more code than its
        // exact waits gain)
        auto sub_chunk = [&](int js, auto refill) {
            const int len = min(SUB, j1 - js);
            const int jn = js + SUB, lenn = min(SUB, j1 - jn);   // the next sub-chunk
            // scores (q is read from LDS; all lanes take part in the lane sums)
            {
#pragma unroll
                for (int t = 0; t < NG; ++t) {
                    const int jl = jloc(t);
                    const u32x4 kv = js + jl == pnew ? knew : kr[t];
                    const float kf[8] = {bf_lo(kv.x), bf_hi(kv.x), bf_lo(kv.y), bf_hi(kv.y),
                                         bf_lo(kv.z), bf_hi(kv.z), bf_lo(kv.w), bf_hi(kv.w)};
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
                        if (jl < len && (lane % LP) == 0) sp[h * SUB + jl] = s * scale;
                    }
                }
            }
            if (bool(refill)) issue_one(kr, Kb, jn, lenn);
            lds_barrier();
            // softmax statistics: wave h owns head h
            if (wid < G) {
                const int h = wid;
                float mx = -INFINITY;
                for (int j = lane; j < len; j += 64) mx = fmaxf(mx, sp[h * SUB + j]);
                mx = wave_max(mx);
                const float mold = st[h * 4], mnew = fmaxf(mold, mx);
                const float resc = (mold == -INFINITY) ? 0.f : expf(mold - mnew);
                float sum = 0.f;
                for (int j = lane; j < len; j += 64) {
                    const float e = expf(sp[h * SUB + j] - mnew);
                    sp[h * SUB + j] = e;
                    sum += e;
                }
                sum = wave_sum(sum);
                if (lane == 0) {
                    st[h * 4 + 0] = mnew;
                    st[h * 4 + 1] = st[h * 4 + 1] * resc + sum;
                    st[h * 4 + 2] = resc;
                }
            }
            lds_barrier();
            // values
            {
#pragma unroll
                for (int h = 0; h < G; ++h) {
                    const float r = st[h * 4 + 2];
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[h][e] *= r;
                }
#pragma unroll
                for (int t = 0; t < NG; ++t) {
                    const int jl = jloc(t);
                    if (jl < len) {
                        const u32x4 vv = js + jl == pnew ? vnew : vr[t];
                        const float vf[8] = {bf_lo(vv.x), bf_hi(vv.x), bf_lo(vv.y), bf_hi(vv.y),
                                             bf_lo(vv.z), bf_hi(vv.z), bf_lo(vv.w), bf_hi(vv.w)};
#pragma unroll
                        for (int h = 0; h < G; ++h) {
                            const float pr = sp[h * SUB + jl];
#pragma unroll
                            for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pr, vf[e], acc[h][e]);
                        }
                    }
                }
            }
            if (bool(refill)) issue_one(vr, Vb, jn, lenn);
            lds_barrier();
        };
        for (int js = j0; js < j1; js += SUB) sub_chunk(js, js + SUB < j1);
    }
    // reduce the PP position slots of each wave, then the waves in order
    if (compute) {
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
    }
    lds_barrier();
    // publish: unnormalised outputs [G][D] and (max, sum) per head
    {
        // tagged words, per query head h: outputs, max, sum (D + 2 words at
        // [b][g][h][c]: the chunks of one query head are contiguous for the
        // O projection, which polls them; no drain, no counter)
        const unsigned tag = ll_tag(P, l);
        unsigned long long *out = P.po_ll + (((size_t)b * P.nkv + g) * G * P.C + c) * (D + 2);
        const size_t hstride = (size_t)P.C * (D + 2);
        for (int t = kl_tid(); t < G * D; t += kThreads) {
            const int h = t / D, dd = t % D;
            float s = 0.f;
            for (int w = 0; w < kWaves; ++w) s += red[(w * G + h) * D + dd];
            st_ll_f(out + h * hstride + dd, s, tag);
        }
        if (kl_tid() < G) {
            st_ll_f(out + kl_tid() * hstride + D, st[kl_tid() * 4 + 0], tag);
            st_ll_f(out + kl_tid() * hstride + D + 1, st[kl_tid() * 4 + 1], tag);
        }
    }
    if (is_ctl_lane0()) trace_stamp(P, ti, 3);
    lds_barrier();   // (the attention area is the next item's)
}


// Streaming attention item (batched path, where an item is a whole sequence
// or a long chunk of one): each compute
// wave streams its own slabs of the chunk (slabs w, w + kWaves, ...; a slab
// is PP positions, one 16-byte load per lane) through a ring of kAttnRing K
// and kAttnRing V loads that is refilled as it is consumed, and each lane
// group (the LP lanes of one position) keeps its own running softmax per
// query head: max m, sum l and the unnormalised output over its 8 dims,
// updated once per kAttnRing slabs (their scores first, one rescale by
// 2^(m_old - m_new) when the max grows, then their values; scores are kept
// in log2 units, so every weight is one hardware exp2).  No block barrier in
// the loop: the PP lane groups of a wave are merged by shuffles, the waves in
// order through LDS.  The queries are held in registers.  The new slot
// (written this step by another workgroup) is read after the wait with
// device-coherent loads into LDS and taken from there; its ring load targets
// a shared dummy line.  Outputs as attn_item's batched path: the chunk's
// (max, sum, unnormalised output), and the normalised output when the item is
// the whole sequence.
template <int D, int G, bool LL>
__device__ __forceinline__ void attn_item_stream(KArg ka, int l, int b, int g, int c, bool first,
                                                 int ti) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    constexpr int LP = D / 8;                       // lanes per position
    constexpr int PP = 64 / LP;                     // positions per slab
    constexpr int R = kAttnRing;
    // Batched path, D = 128: the scores of a ring round (R slabs of PP
    // positions, 16 rows) are one v_mfma_f32_16x16x32_bf16 tile per 32
    // columns, the K rows as A and the team's queries (scaled, as two bf16
    // terms) as B.  The K ring then holds A-operand pieces: load ks of a
    // round is columns 32 ks + 8 (l / 16) .. + 7 of tile row l % 16 (slab
    // (l % 16) / PP, position (l % 16) % PP).  The tile goes through a
    // per-wave LDS slot to the lanes of its positions; the softmax and the
    // values stay on the vector units.  (Step time, same device: 8B shape,
    // batch 32, 8.07 -> 7.97 ms; 70B shape, batch 32, 47.1-47.8 -> 46.3-46.7
    // ms.  The per-sequence path's chunks are a few rounds long, where the
    // vector-unit scores measured faster: 70B shape, batch 1, 23.8 against
    // 24.2 ms.)
    constexpr bool MC = D == 128 && !LL;
    static_assert(!MC || (R * PP == 16 && R * 32 == D), "one 16-row tile per ring round");
    // more than 4 query heads per KV head: the waves split into NH teams of
    // HG heads each; every team streams the whole chunk (the second team's
    // loads of the same lines meet them in L2)
    constexpr int HG = G < 4 ? G : 4, NH = G / HG, TW = kWaves / NH;
    static_assert(G % HG == 0 && kWaves % NH == 0, "head teams");
    const int wid = __builtin_amdgcn_readfirstlane(kl_tid() >> 6);
    const int team = wid / TW, tw = wid % TW;      // (the control wave: team NH)
    const int h0 = team * HG;                      // the team's first query head
    const int lane = kl_tid() & 63;
    const int pi = lane / LP, ds = (lane % LP) * 8;
    const int pnew = pos_of<LL>(P, b), n = pnew + 1;
    int s0, s1;
    split_range((n + PP - 1) / PP, P.C, c, s0, s1);
    const bool compute = wid < kWaves;
    // this wave's slabs: s0 + tw, s0 + tw + TW, ... < s1
    const int mine = compute && s0 + tw < s1 ? (s1 - s0 - tw + TW - 1) / TW : 0;

    float *qs = S.attn;                                  // [G][D]
    float *wm = qs + G * D;                              // [kWaves][HG] wave maxima (log2 units)
    float *wl = wm + kWaves * HG;                        // [kWaves][HG] wave sums
    float *wacc = wl + kWaves * HG;                      // [kWaves][HG][D] wave outputs
    uint16_t *kn = reinterpret_cast<uint16_t *>(wacc + kWaves * HG * D);  // [D] new key
    uint16_t *vn = kn + D;                                                // [D] new value
    float *stile = reinterpret_cast<float *>(vn + D) + min(wid, kWaves - 1) * 256;   // [16][16]
    const size_t row0 = kv_row(P, l, b, g);
    const uint16_t *Kb = P.kc + row0 * D + ds;
    const uint16_t *Vb = P.vc + row0 * D + ds;
    // scores in log2 units: softmax weights are 2^(s log2(e) - max)
    const float scale = 1.4426950408889634f / sqrtf((float)D);

    // the ring: item i of this wave (slab s0 + wid + i kWaves) sits in slot
    // i % R; a slot past the wave's slabs, past the context or holding the
    // new position loads the dummy line (zeros)
    u32x4 kr[R], vr[R];
    auto pos_of_item = [&](int i) { return (s0 + tw + i * TW) * PP + pi; };
    // MC: this lane's tile row (slab ksl, position kpi) and columns
    const int ksl = (lane & 15) / PP, kpi = (lane & 15) % PP, kcol = 8 * (lane >> 4);
    auto kpos = [&](int i0) { return (s0 + tw + (i0 + ksl) * TW) * PP + kpi; };
    auto kaddr = [&](int i0, int ks) -> const void * {
        const int pos = kpos(i0);
        return (i0 + ksl < mine && pos < n && pos != pnew)
                   ? (const void *)(P.kc + (row0 + pos) * D + 32 * ks + kcol)
                   : (const void *)P.dummy;
    };
    auto addr = [&](const uint16_t *base, int i) -> const void * {
        const int pos = pos_of_item(i);
        return (i < mine && pos < n && pos != pnew) ? (const void *)(base + (size_t)pos * D)
                                                    : (const void *)P.dummy;
    };
    if (compute) {
#pragma unroll
        for (int s = 0; s < R; ++s) kr[s] = ld_stream_16B(MC ? kaddr(0, s) : addr(Kb, s));
#pragma unroll
        for (int s = 0; s < R; ++s) vr[s] = ld_stream_16B(addr(Vb, s));
    }
    if (is_ctl_lane0()) trace_stamp(P, ti, 1);
    if constexpr (LL) {
        // the queries of head g's query heads and the new key and value, as
        // tagged words (every thread takes a few), into LDS
        const size_t qo = (size_t)b * P.nq * D + (size_t)g * G * D;
        const unsigned long long *kvl = P.kv_ll + ((size_t)b * P.nkv + g) * D;
        ll_gather<(G * D + D + kThreads - 1) / kThreads>(
            P, G * D + D, ll_tag(P, l), kl_tid(), kThreads,
            [&](int i) { return i < G * D ? P.q_ll + qo + i : kvl + (i - G * D); },
            [&](int i, unsigned v) {
                if (i < G * D) {
                    qs[i] = __uint_as_float(v);
                } else if (i < G * D + D / 2) {   // key dims j and j + D/2
                    const int j = i - G * D;
                    kn[j] = (uint16_t)v;
                    kn[j + D / 2] = (uint16_t)(v >> 16);
                } else {                           // value dims 2j and 2j + 1
                    reinterpret_cast<unsigned *>(vn)[i - G * D - D / 2] = v;
                }
            });
    } else {
        if (first) local_wait(P, P.cnt + g, (unsigned)(l + 1) * (unsigned)P.Sg, ti);
        // the queries and the new key and value (device-coherent loads, all
        // unconditional from clamped addresses and issued together; masked
        // when stored)
        constexpr int NQ = (G * D + kThreads - 1) / kThreads;
        float qv[NQ];
        const float *qsrc = P.q + (size_t)b * P.nq * D + (size_t)g * G * D;
#pragma unroll
        for (int k = 0; k < NQ; ++k) qv[k] = ld_dev(qsrc + min((int)kl_tid() + k * kThreads, G * D - 1));
        const size_t o = (size_t)pnew * D + min((int)kl_tid(), D / 4 - 1) * 4;
        const unsigned long long kw = ld_dev_u64(P.kc + row0 * D + o);
        const unsigned long long vw = ld_dev_u64(P.vc + row0 * D + o);
#pragma unroll
        for (int k = 0; k < NQ; ++k)
            if ((int)kl_tid() + k * kThreads < G * D) qs[kl_tid() + k * kThreads] = qv[k];
        if (kl_tid() < D / 4) {
            reinterpret_cast<unsigned long long *>(kn)[kl_tid()] = kw;
            reinterpret_cast<unsigned long long *>(vn)[kl_tid()] = vw;
        }
    }
    __syncthreads();
    if (is_ctl_lane0()) trace_stamp(P, ti, 2);

    float acc[HG][8], m[HG], lsum[HG];
#pragma unroll
    for (int h = 0; h < HG; ++h) {
        m[h] = -INFINITY;
        lsum[h] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    }
    if (compute) {
        float q[MC ? 1 : HG][8];
        bf16x8 qb[MC ? R : 1], qbl[MC ? R : 1];
        if constexpr (MC) {
            // B operand: column l % 16 = the team's head l % 16 (zero past HG)
            const int hc = lane & 15;
#pragma unroll
            for (int ks = 0; ks < R; ++ks) {
                unsigned hw[4], lw[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int d0 = 32 * ks + kcol + 2 * j;
                    const float x0 = hc < HG ? qs[(h0 + hc) * D + d0] * scale : 0.f;
                    const float x1 = hc < HG ? qs[(h0 + hc) * D + d0 + 1] * scale : 0.f;
                    split_bf16x2(x0, x1, hw[j], lw[j]);
                }
                qb[ks] = __builtin_bit_cast(bf16x8, u32x4{hw[0], hw[1], hw[2], hw[3]});
                qbl[ks] = __builtin_bit_cast(bf16x8, u32x4{lw[0], lw[1], lw[2], lw[3]});
            }
        } else {
#pragma unroll
            for (int h = 0; h < HG; ++h) {
                const float4 q0 = *reinterpret_cast<const float4 *>(qs + (h0 + h) * D + ds);
                const float4 q1 = *reinterpret_cast<const float4 *>(qs + (h0 + h) * D + ds + 4);
                q[h][0] = q0.x; q[h][1] = q0.y; q[h][2] = q0.z; q[h][3] = q0.w;
                q[h][4] = q1.x; q[h][5] = q1.y; q[h][6] = q1.z; q[h][7] = q1.w;
            }
        }
        // R slabs at a time: their scores, one rescale per head, their values
        for (int i0 = 0; i0 < mine; i0 += R) {
            float sc[R][HG];
            if constexpr (MC) {
                const bool knew = kpos(i0) == pnew;   // (the new key comes from LDS)
                f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < R; ++ks) {
                    const u32x4 kv = knew ? *reinterpret_cast<const u32x4 *>(kn + 32 * ks + kcol)
                                          : kr[ks];
                    kr[ks] = ld_stream_16B(kaddr(i0 + R, ks));
                    const bf16x8 a = __builtin_bit_cast(bf16x8, kv);
                    t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qb[ks], t, 0, 0, 0);
                    t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qbl[ks], t, 0, 0, 0);
                }
                // D lane l: rows 4 (l / 16) + v, column l % 16 (wave-local slot:
                // a wave's LDS accesses complete in order)
#pragma unroll
                for (int v = 0; v < 4; ++v) stile[(4 * (lane >> 4) + v) * 16 + (lane & 15)] = t[v];
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
                for (int s = 0; s < R; ++s) {
                    const int pos = pos_of_item(i0 + s);
                    const bool valid = i0 + s < mine && pos < n;
                    const float4 v4 = *reinterpret_cast<const float4 *>(stile + (s * PP + pi) * 16);
                    const float vv[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
                    for (int h = 0; h < HG; ++h) sc[s][h] = valid ? vv[h] : -INFINITY;
                }
            } else {
#pragma unroll
                for (int s = 0; s < R; ++s) {
                    const int pos = pos_of_item(i0 + s);
                    const bool valid = i0 + s < mine && pos < n;
                    const u32x4 kv =
                        pos == pnew ? *reinterpret_cast<const u32x4 *>(kn + ds) : kr[s];
                    kr[s] = ld_stream_16B(addr(Kb, i0 + s + R));
                    const float kf[8] = {bf_lo(kv.x), bf_hi(kv.x), bf_lo(kv.y), bf_hi(kv.y),
                                         bf_lo(kv.z), bf_hi(kv.z), bf_lo(kv.w), bf_hi(kv.w)};
#pragma unroll
                    for (int h = 0; h < HG; ++h) {
                        float d = 0.f;
#pragma unroll
                        for (int e = 0; e < 8; ++e) d = fmaf(q[h][e], kf[e], d);
                        d = sum_lanes<LP>(d) * scale;
                        sc[s][h] = valid ? d : -INFINITY;
                    }
                }
            }
#pragma unroll
            for (int h = 0; h < HG; ++h) {
                float mx = m[h];
#pragma unroll
                for (int s = 0; s < R; ++s) mx = fmaxf(mx, sc[s][h]);
                const float al = m[h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[h] - mx);
                float sum = 0.f;
#pragma unroll
                for (int s = 0; s < R; ++s) {
                    sc[s][h] = sc[s][h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[s][h] - mx);
                    sum += sc[s][h];
                }
                lsum[h] = fmaf(lsum[h], al, sum);
                m[h] = mx;
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h][e] *= al;
            }
#pragma unroll
            for (int s = 0; s < R; ++s) {
                const int pos = pos_of_item(i0 + s);
                const u32x4 vv = pos == pnew ? *reinterpret_cast<const u32x4 *>(vn + ds) : vr[s];
                vr[s] = ld_stream_16B(addr(Vb, i0 + s + R));
                const float vf[8] = {bf_lo(vv.x), bf_hi(vv.x), bf_lo(vv.y), bf_hi(vv.y),
                                     bf_lo(vv.z), bf_hi(vv.z), bf_lo(vv.w), bf_hi(vv.w)};
#pragma unroll
                for (int h = 0; h < HG; ++h)
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(sc[s][h], vf[e], acc[h][e]);
            }
        }
        // merge the PP lane groups of the wave (lanes ds apart by LP, 2 LP, ...)
#pragma unroll
        for (int off = LP; off < 64; off <<= 1) {
#pragma unroll
            for (int h = 0; h < HG; ++h) {
                const float m2 = __shfl_xor(m[h], off), l2 = __shfl_xor(lsum[h], off);
                const float mn = fmaxf(m[h], m2);
                const float a1 = m[h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[h] - mn);
                const float a2 = m2 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m2 - mn);
                lsum[h] = lsum[h] * a1 + l2 * a2;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float o2 = __shfl_xor(acc[h][e], off);
                    acc[h][e] = acc[h][e] * a1 + o2 * a2;
                }
                m[h] = mn;
            }
        }
        if (pi == 0) {
#pragma unroll
            for (int h = 0; h < HG; ++h) {
#pragma unroll
                for (int e = 0; e < 8; ++e) wacc[(wid * HG + h) * D + ds + e] = acc[h][e];
                if (ds == 0) {
                    wm[wid * HG + h] = m[h];
                    wl[wid * HG + h] = lsum[h];
                }
            }
        }
    }
    __syncthreads();
    // the waves in order: (max, sum, unnormalised output) of the chunk, the
    // max published in natural-log units; per-sequence path: as tagged
    // words, per query head h at [b][g][h][c] (D + 2 words: outputs, max,
    // sum; one query head's chunks contiguous for the O projection, which
    // polls them)
    const size_t item = ((size_t)b * P.nkv + g) * P.C + c;
    float *out = P.part_o + item * G * D;
    float *sts = P.part_s + item * G * 2;
    unsigned long long *ll_out = P.po_ll + (((size_t)b * P.nkv + g) * G * P.C + c) * (D + 2);
    const size_t hstride = (size_t)P.C * (D + 2);
    const unsigned tag = ll_tag(P, l);
    for (int t = kl_tid(); t < G * D + G; t += kThreads) {
        const int h = t < G * D ? t / D : t - G * D, dd = t % D;
        const int w0 = (h / HG) * TW, hl = h % HG;   // the head's team, its slot
        float M = -INFINITY;
        for (int w = w0; w < w0 + TW; ++w) M = fmaxf(M, wm[w * HG + hl]);
        float O = 0.f, L = 0.f;
        for (int w = w0; w < w0 + TW; ++w) {
            const float mw = wm[w * HG + hl];
            const float a = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - M);
            L = fmaf(wl[w * HG + hl], a, L);
            if (t < G * D) O = fmaf(wacc[(w * HG + hl) * D + dd], a, O);
        }
        if constexpr (LL) {
            if (t < G * D) {
                st_ll_f(ll_out + h * hstride + dd, O, tag);
            } else {
                st_ll_f(ll_out + h * hstride + D, M * 0.6931471805599453f, tag);
                st_ll_f(ll_out + h * hstride + D + 1, L, tag);
            }
        } else if (t < G * D) {
            st_dev(out + t, O);
            if (P.C == 1) {   // (one chunk: the merged output is final)
                uint16_t hi, lo;
                split_bf16(O / L, hi, lo);
                const size_t o = (size_t)b * P.nq * D + (size_t)g * G * D + t;
                st_dev_u16(P.acto + o, hi);
                st_dev_u16(P.acto_lo + o, lo);
            }
        } else {
            st_dev(sts + h * 2, M * 0.6931471805599453f);
            st_dev(sts + h * 2 + 1, L);
        }
    }
    if (is_ctl_lane0()) trace_stamp(P, ti, 3);
    __syncthreads();   // (the attention area is the next item's)
}

// Attention of KV head g: the workgroups of head g take its items (sequence
// b, chunk c) round-robin.  The per-sequence path hands the chunk results to
// the O projection as tagged words; the batched path publishes them before a
// grid barrier.
template <int D, int G, bool BAT>
__device__ __forceinline__ void phase_attn(KArg ka, int l, int garrive, int ti) {
    const StepParams P = load_params(ka);
    const int g = blockIdx.x / P.Sg, part = blockIdx.x % P.Sg;
    if (g < P.nkv) {
        const int items = P.B * P.C;
        for (int it = part; it < items; it += P.Sg)
            if constexpr (!BAT && G <= 4)
                attn_item_ll<D, G>(ka, l, it / P.C, g, it % P.C, ti);
            else
                attn_item_stream<D, G, !BAT>(ka, l, it / P.C, g, it % P.C, it == part, ti);
    }
    if (garrive >= 0) bar_arrive(P, garrive, ti);
    else if (is_ctl_lane0()) trace_stamp(P, ti, 0);
}

// O projection of KV head g: x += Wo[:, columns of head g] o_g, for the rows
// this workgroup owns among head g's workgroups, added into the fixed-point
// residual.  GEMV path: the staged input is head g's merged attention output,
// published by the attention phase.
template <int D, int G, bool BAT>
__device__ __forceinline__ void phase_oproj(KArg ka, int l, int gwait, int mbar, int garrive,
                                            int ti) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    const int KTO = G * D / kTileK;
    const uint8_t *Wo = P.arena + (size_t)l * P.layer_stride + P.off_o;
    auto epi = [&](int b, int r, float y0, float y1) {
        long long *x = P.xf + (size_t)b * P.Hp;
        add_fix(x + r, y0);
        add_fix(x + r + 1, y1);
    };
    if constexpr (BAT) {
        // 2-D partition: KSo K slices (the columns of nkv / KSo KV heads
        // each) x row groups; a workgroup writes its slice's partial sums,
        // which the next RMSNorm step folds into the residual.  Every wave
        // gets whole 16-row blocks and the activation staging is one slice.
        // (The O projection is packed per query head, D / kTileK k-tiles per
        // row group: a slice spans gps G packed matrices.)
        const int KS = P.KSo, RB = P.nwg / KS;
        const int ks = blockIdx.x / RB, rb = blockIdx.x % RB, ksc = min(ks, KS - 1);
        const int gps = P.nkv / KS, width = gps * G * D;   // KV heads and columns per slice
        int a0 = 0, a1 = 0;
        if (ks < KS) split_range(P.o_rg, RB, rb, a0, a1);
        const int col0 = ksc * width;
        float *part = P.xpart + (size_t)ksc * P.xpart_stride;
        weight_phase<true>(
            P, S, Wo + (size_t)ksc * gps * P.o_rg * KTO * kTileBytes, gps * KTO, a0, a1 - a0,
            [&]() { if (gwait >= 0) bar_wait(P, gwait, ti); },
            [&]() { if (mbar >= 0) merge_batched<D, G>(P, mbar); }, [&](int) {},
            [&](int c, int b0, int nb, uint16_t *buf) {
                stage_bf16_chunk(P.acto + col0, P.acto_lo + col0, P.nq * D, width, c, b0, nb, buf);
            },
            [&](int b, int r, float y0, float y1) {
                st_dev(part + (size_t)b * P.Hp + r, y0);
                st_dev(part + (size_t)b * P.Hp + r + 1, y1);
            },
            D / kTileK, (size_t)P.o_rg * (D / kTileK));
    } else {
        // per query head: the Sg workgroups of KV head g split into G
        // groups, group hq applying the O-projection columns of query head
        // g G + hq to its merged attention output, each workgroup for a
        // range of rows
        const int g = blockIdx.x / P.Sg, part = blockIdx.x % P.Sg;
        if (g < P.nkv) {
            int hq = 0;
            while (hq + 1 < G && part >= (P.Sg * (hq + 1)) / G) ++hq;
            const int p0 = (P.Sg * hq) / G, np = (P.Sg * (hq + 1)) / G - p0;
            int a0, a1;
            split_range(P.o_rg, np, part - p0, a0, a1);
            constexpr int KTq = D / kTileK;
            // With up to 4 query heads per KV head the waves split: waves
            // kOEarly .. kWaves - 1 issue their loads before the merge and take
            // no part in its gather, so half the matrix streams while the merge
            // waits for the attention's chunks; waves 0 .. kOEarly - 1 gather
            // the chunks and issue their loads after the merge.  (Every wave
            // issuing its loads first makes the merge's gather queue behind
            // them; the control wave in the gather slows it.)  The early waves
            // go early only when one ring holds their whole share (at 8 query
            // heads per KV head the share is several rings, and the split was
            // measured slower).
            constexpr bool SPLIT = G <= 4;
            constexpr int NTM = SPLIT ? kOEarly * 64 : kThreads;
            const int mine = ((a1 - a0) + kWaves - 1) / kWaves * KTq;   // tiles per wave, at most
            const int EW = SPLIT && mine <= kGemvDepth ? kOEarly : kWaves + 1;
            auto stage = [&](int b) {
                if (b == 0 && is_ctl_lane0()) trace_stamp(P, ti, 1);
                // (with P.multi sequence b's output goes to S.a + b D; all
                // sequences in one gather when their chunks fit)
                if (!P.multi)
                    merge_ll<D, G, NTM>(P, l, b, g, hq, S.a, S.a + D);
                else if (P.B * P.C > kMergeChunks)
                    merge_ll<D, G, NTM>(P, l, b, g, hq, S.a + b * D, S.a + kMultiSeq * D);
                else if (b == 0)
                    merge_ll_multi<D, G, NTM>(P, l, P.B, g, hq, S);
                if (b == 0 && is_ctl_lane0()) {
                    trace_stamp(P, ti, 2);
                    trace_stamp(P, ti, 3);
                }
            };
            const uint8_t *W = Wo + (size_t)(g * G + hq) * P.o_rg * KTq * kTileBytes;
            if (P.multi)
                gemv_phase<false, SPLIT, true>(W, KTq, a0, a1 - a0, 1, P.B, S.a, S.red, P.dummy,
                                               [&]() {}, stage, epi, EW, D);
            else
                gemv_phase<false, SPLIT>(W, KTq, a0, a1 - a0, 1, P.B, S.a, S.red, P.dummy,
                                         [&]() {}, stage, epi, EW);
        }
    }
    if (garrive >= 0) bar_arrive(P, garrive, ti);
}


// ---------------------------------------------------------------- mixture of experts
//
// Per-sequence path (the Mixtral variant of Table 2).  Each of a token's
// top_k expert slots has nwg / top_k workgroups, laid out like the dense
// FFN's (column block j = w / Rc of the slot's expert).  Every workgroup
// computes the router logits of every sequence itself (same data, same
// order: the same values everywhere), so no hand-off is needed, and keeps
// the chosen experts in LDS for the down phase of the same launch.

// Router logits of sequence b from the staged activation (a = x gain, the
// RMSNorm scale deferred as in the gate/up product): the packed router (one
// row group of E <= 8 rows) split over the compute waves by k-tiles, the
// wave partials added in wave order; then the top_k experts (the lowest index
// first among equal logits) and the softmax of their logits.
__device__ __forceinline__ void route_experts(const StepParams &P, const Lds &S,
                                              const uint8_t *Lb, int b) {
    const int wid = __builtin_amdgcn_readfirstlane(kl_tid() >> 6);
    const int lane = kl_tid() & 63, row = lane >> 3, sub = lane & 7;
    const int KT = P.Hp / kTileK;
    if (wid < kWaves) {
        const uint8_t *R = Lb + P.off_router + (size_t)lane * 16;
        float acc = 0.f;
        for (int kt = (wid * KT) / kWaves; kt < ((wid + 1) * KT) / kWaves; ++kt) {
            const u32x4 w = *reinterpret_cast<const u32x4 *>(R + (size_t)kt * kTileBytes);
            const float *ap = S.a + kt * kTileK + sub * 8;
            const float4 a0 = *reinterpret_cast<const float4 *>(ap);
            const float4 a1 = *reinterpret_cast<const float4 *>(ap + 4);
            acc = fmaf(bf_lo(w.x), a0.x, acc);
            acc = fmaf(bf_hi(w.x), a0.y, acc);
            acc = fmaf(bf_lo(w.y), a0.z, acc);
            acc = fmaf(bf_hi(w.y), a0.w, acc);
            acc = fmaf(bf_lo(w.z), a1.x, acc);
            acc = fmaf(bf_hi(w.z), a1.y, acc);
            acc = fmaf(bf_lo(w.w), a1.z, acc);
            acc = fmaf(bf_hi(w.w), a1.w, acc);
        }
        acc = sum8(acc);
        if (sub == 0) S.red[wid * kTileRows + row] = acc;
    }
    lds_barrier();
    float *logit = S.red + kWaves * kTileRows;
    if (kl_tid() < kTileRows) {
        float t = 0.f;
        for (int w = 0; w < kWaves; ++w) t += S.red[w * kTileRows + kl_tid()];
        logit[kl_tid()] = t * rms_scale(S.sm, P.H, P.eps);
    }
    lds_barrier();
    if (kl_tid() == 0) {
        int e0 = 0;
        for (int e = 1; e < P.E; ++e)
            if (logit[e] > logit[e0]) e0 = e;
        int e1 = e0;
        float w0 = 1.f, w1 = 0.f;
        if (P.topk == 2) {
            e1 = -1;
            for (int e = 0; e < P.E; ++e)
                if (e != e0 && (e1 < 0 || logit[e] > logit[e1])) e1 = e;
            const float t = expf(logit[e1] - logit[e0]);   // softmax of the two logits
            w0 = 1.f / (1.f + t);
            w1 = t / (1.f + t);
        }
        int *rt = route_table(P) + 4 * b;
        rt[0] = e0;
        rt[1] = e1;
        rt[2] = __float_as_int(w0);
        rt[3] = __float_as_int(w1);
    }
    lds_barrier();
}

// The expert slot, FFN column block and part of this workgroup (slot >= topk
// or j >= Sc: no FFN rows).
struct MoeShare { int slot, j, part; };
__device__ __forceinline__ MoeShare moe_share(const StepParams &P) {
    const int nwk = P.nwg / P.topk, loc = blockIdx.x % nwk;
    return MoeShare{(int)blockIdx.x / nwk, loc / P.Rc, loc % P.Rc};
}

// RMSNorm, router, and the gate/up product + SwiGLU of this workgroup's
// expert slot for each sequence: m[b][slot] as tagged words.
__device__ __forceinline__ void moe_gateup(const StepParams &P, const Lds &S, int l, int gwait,
                                           int ti) {
    const uint8_t *Lb = P.arena + (size_t)l * P.layer_stride;
    const float *gain = reinterpret_cast<const float *>(Lb + P.off_ffn_norm);
    const MoeShare ms = moe_share(P);
    const bool member = ms.slot < P.topk && ms.j < P.Sc;
    int first = 0, count = 0;
    if (member) {   // as the dense FFN: block j covers SwiGLU outputs [j KTc 64, + KTc 64)
        const int r0 = min(P.gu_rg, ms.j * P.KTc * 2 * kTileK / kTileRows);
        const int r1 = min(P.gu_rg, (ms.j + 1) * P.KTc * 2 * kTileK / kTileRows);
        int a0, a1;
        split_range(r1 - r0, P.Rc, ms.part, a0, a1);
        first = r0 + a0;
        count = a1 - a0;
    }
    if (gwait >= 0) bar_wait(P, gwait, ti);
    for (int b = 0; b < P.B; ++b) {
        stage_rms_deferred(P.xf + (size_t)b * P.Hp, gain, P.H, P.Hp, S.a, S.sm);
        route_experts(P, S, Lb, b);
        if (b == 0 && is_ctl_lane0()) trace_stamp(P, ti, 3);
        const int e = member ? route_table(P)[4 * b + ms.slot] : 0;
        gemv_phase<true>(
            Lb + P.off_gu + (size_t)e * P.gu_estride, P.Hp / kTileK, first, count, 1, 1, S.a,
            S.red, P.dummy, [&]() {}, [&](int) {},
            [&](int, int r, float gt, float up) {
                const float rs = rms_scale(S.sm, P.H, P.eps);
                gt *= rs;
                up *= rs;
                st_ll_f(P.m_ll + ((size_t)b * P.topk + ms.slot) * P.Fp + (r >> 1),
                        gt / (1.0f + expf(-gt)) * up, ll_tag(P, l));
            });
    }
}

// Down product of this workgroup's expert slot for each sequence, weighted
// by the slot's router weight, added into the residual.
__device__ __forceinline__ void moe_down(const StepParams &P, const Lds &S, int l, int ti) {
    const MoeShare ms = moe_share(P);
    if (ms.slot >= P.topk || ms.j >= P.Sc) return;
    int a0, a1;
    split_range(P.down_rg, P.Rc, ms.part, a0, a1);
    const int kw = P.KTc * kTileK, c0 = ms.j * kw, nreal = max(0, min(kw, P.F - c0));
    for (int b = 0; b < P.B; ++b) {
        const int *rt = route_table(P) + 4 * b;
        const int e = rt[ms.slot];
        const float we = __int_as_float(rt[2 + ms.slot]);
        gemv_phase<true>(
            P.arena + (size_t)l * P.layer_stride + P.off_down + (size_t)e * P.down_estride +
                (size_t)ms.j * P.down_rg * P.KTc * kTileBytes,
            P.KTc, a0, a1 - a0, 1, 1, S.a, S.red, P.dummy, [&]() {},
            [&](int) {
                if (b == 0 && is_ctl_lane0()) trace_stamp(P, ti, 1);
                if ((kl_tid() >> 6) == kCtlWave)
                    ll_gather<kDownGather>(
                        P, nreal, ll_tag(P, l), kl_tid() & 63, 64,
                        [&](int i) {
                            return P.m_ll + ((size_t)b * P.topk + ms.slot) * P.Fp + c0 + i;
                        },
                        [&](int i, unsigned v) { S.a[i] = __uint_as_float(v); });
                for (int i = nreal + kl_tid(); i < kw; i += kThreads) S.a[i] = 0.f;
                lds_barrier();
                if (b == 0 && is_ctl_lane0()) {
                    trace_stamp(P, ti, 2);
                    trace_stamp(P, ti, 3);
                }
            },
            [&](int, int r, float y0, float y1) {
                long long *x = P.xf + (size_t)b * P.Hp;
                add_fix(x + r, we * y0);
                add_fix(x + r + 1, we * y1);
            });
    }
}

// RMSNorm + gate/up projection + SwiGLU for FFN column block j = w / Rc:
// m = silu(Wg u) * (Wu u).  Packed rows alternate gate i, up i.
template <bool BAT>
__device__ __forceinline__ void phase_gateup(KArg ka, int l, int gwait, int garrive, int ti) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    const uint8_t *Lb = P.arena + (size_t)l * P.layer_stride;
    const float *gain = reinterpret_cast<const float *>(Lb + P.off_ffn_norm);
    if constexpr (BAT) {
        // 2-D partition: KSg K slices (of Hp / KSg columns, one chunk or a
        // few) x row groups, so a workgroup's load ring streams through all
        // of its blocks within few chunks; the gate and up partial sums go
        // to the slice's partial buffer, and the SwiGLU is applied when the
        // down phase folds them (fold_swiglu)
        const int KS = P.KSg, RB = P.nwg / KS, KT = P.Hp / kTileK, KTs = KT / KS;
        const int ks = blockIdx.x / RB, rb = blockIdx.x % RB, ksc = min(ks, KS - 1);
        int a0 = 0, a1 = 0;
        if (ks < KS) split_range(P.gu_rg, RB, rb, a0, a1);
        const int col0 = ksc * KTs * kTileK;
        float *part = P.gpart + (size_t)ksc * P.gpart_stride;
        const int grow = P.gu_rg * kTileRows;
        weight_phase<true>(
            P, S, Lb + P.off_gu + (size_t)ksc * KTs * kTileBytes, KTs, a0, a1 - a0,
            [&]() { if (gwait >= 0) bar_wait(P, gwait, ti); },
            // (folds the O projection's partials, x: xf -> xf2)
            [&]() {
                norm_batched(P, S, gain, P.xf, P.xf2, P.KSo);
                if (is_ctl_lane0()) trace_stamp(P, ti, 3);
            },
            [&](int) {},
            [&](int c, int b0, int nb, uint16_t *buf) {
                const int sl = col0 / kGemmChunkK + c;
                if (b0 == 0) norm_wait(P, 2 * l + 1, sl, sl + 1);
                stage_bf16_chunk(P.act + col0, P.act_lo + col0, P.Hp, KTs * kTileK, c, b0, nb, buf);
            },
            [&](int b, int r, float gt, float up) {
                st_dev(part + (size_t)b * grow + r, gt);
                st_dev(part + (size_t)b * grow + r + 1, up);
            },
            KT, 0);
        if (garrive >= 0) bar_arrive(P, garrive, ti);
        return;
    }
    if (P.E > 1) {
        moe_gateup(P, S, l, gwait, ti);
        if (is_ctl_lane0()) trace_stamp(P, ti, 0);
        return;
    }
    const int j = blockIdx.x / P.Rc, part = blockIdx.x % P.Rc;
    const bool member = j < P.Sc;
    int first = 0, count = 0;
    if (member) {
        // block j covers SwiGLU outputs [j KTc 64, (j + 1) KTc 64): 2 packed rows each
        const int r0 = min(P.gu_rg, j * P.KTc * 2 * kTileK / kTileRows);
        const int r1 = min(P.gu_rg, (j + 1) * P.KTc * 2 * kTileK / kTileRows);
        int a0, a1;
        split_range(r1 - r0, P.Rc, part, a0, a1);
        first = r0 + a0;
        count = a1 - a0;
    }
    weight_phase<false>(
        P, S, Lb + P.off_gu, P.Hp / kTileK, first, count,
        [&]() { if (gwait >= 0) bar_wait(P, gwait, ti); }, [&]() {},
        [&](int b) {
            if (P.multi) {
                if (b == 0)
                    stage_rms_multi(P.xf, P.Hp, gain, P.H, P.Hp, P.B, S.a, P.Hp, S.sm, NoExtra(),
                                    NoExtra(), 0);
            } else {
                stage_rms_deferred(P.xf + (size_t)b * P.Hp, gain, P.H, P.Hp, S.a, S.sm);
            }
            if (b == 0 && is_ctl_lane0()) trace_stamp(P, ti, 3);
        },
        [&](int, int, int, uint16_t *) {},
        [&](int b, int r, float gt, float up) {
            // the deferred RMSNorm scale
            const float rs = rms_scale(seq_sm(P, S, b), P.H, P.eps);
            gt *= rs;
            up *= rs;
            st_ll_f(P.m_ll + (size_t)b * P.Fp + (r >> 1), gt / (1.0f + expf(-gt)) * up,
                    ll_tag(P, l));
        },
        0, 0, NoGroupDone(), P.Hp);
    // (the down projection polls the tagged words: no drain, no counter)
    if (is_ctl_lane0()) trace_stamp(P, ti, 0);
}

// Batched path: the SwiGLU of the gate/up K-slice partials, m = silu(g) u with
// g, u the fixed-order sums over the slices, as the two bf16 terms the down
// projection stages; the (sequence, FFN column) elements are spread over the
// grid.  Ends with grid barrier k.
__device__ __forceinline__ void fold_swiglu(const StepParams &P, const Lds &S, int k) {
    const int F = P.F, grow = P.gu_rg * kTileRows, KS = P.KSg;
    rms_table(P, S);
    const int total = P.B * F, stride = P.nwg * kThreads;
    // a thread's elements e0 + k stride, k < FE, are loaded together (one
    // memory round trip per KS / 4 slices instead of one per element)
    constexpr int FE = 4;
    for (int e0 = blockIdx.x * kThreads + kl_tid(); e0 - (int)kl_tid() < total;
         e0 += FE * stride) {
        float gs[FE], us[FE];
#pragma unroll
        for (int k = 0; k < FE; ++k) gs[k] = us[k] = 0.f;
        for (int q0 = 0; q0 < KS; q0 += 4) {
            // (unconditional loads from in-range addresses, masked when used)
            unsigned long long v[FE][4];
#pragma unroll
            for (int k = 0; k < FE; ++k) {
                const int ec = min(e0 + k * stride, total - 1), b = ec / F, f = ec % F;
                const float *src = P.gpart + (size_t)b * grow + 2 * f;
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    v[k][j] = ld_dev_u64(src + (size_t)min(q0 + j, KS - 1) * P.gpart_stride);
            }
#pragma unroll
            for (int k = 0; k < FE; ++k)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (q0 + j < KS) {
                        gs[k] += __uint_as_float((unsigned)v[k][j]);
                        us[k] += __uint_as_float((unsigned)(v[k][j] >> 32));
                    }
                }
        }
#pragma unroll
        for (int k = 0; k < FE; ++k) {
            const int e = e0 + k * stride;
            if (e < total) {
                const int b = e / F, f = e % F;
                const float r = rms_of(P, S, b);   // the deferred RMSNorm scale
                const float g = gs[k] * r, u = us[k] * r;
                uint16_t hi, lo;
                split_bf16(g / (1.0f + expf(-g)) * u, hi, lo);
                st_dev_u16(P.actm + (size_t)b * P.Fp + f, hi);
                st_dev_u16(P.actm_lo + (size_t)b * P.Fp + f, lo);
            }
        }
    }
    bar_arrive(P, k, -1);
    bar_wait(P, k, -1);
}

// Down projection of FFN column block j: x += Wd[:, block j] m[block j], for
// the rows this workgroup owns among block j's workgroups.
template <bool BAT>
__device__ __forceinline__ void phase_down(KArg ka, int l, int gwait, int xbar, int garrive,
                                           int ti) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    const uint8_t *Wd = P.arena + (size_t)l * P.layer_stride + P.off_down;
    auto epi = [&](int b, int r, float y0, float y1) {
        long long *x = P.xf + (size_t)b * P.Hp;
        add_fix(x + r, y0);
        add_fix(x + r + 1, y1);
    };
    if constexpr (BAT) {
        // 2-D partition: KSd K slices (Sc / KSd FFN column blocks each) x row
        // groups, partial sums folded by the next RMSNorm step (as for the O
        // projection)
        const int KS = P.KSd, RB = P.nwg / KS;
        const int ks = blockIdx.x / RB, rb = blockIdx.x % RB, ksc = min(ks, KS - 1);
        const int gps = P.Sc / KS, width = gps * P.KTc * kTileK;
        int a0 = 0, a1 = 0;
        if (ks < KS) split_range(P.down_rg, RB, rb, a0, a1);
        const size_t col0 = (size_t)ksc * width;
        float *part = P.xpart + (size_t)ksc * P.xpart_stride;
        weight_phase<true>(
            P, S, Wd + (size_t)ksc * gps * P.down_rg * P.KTc * kTileBytes, gps * P.KTc, a0,
            a1 - a0, [&]() { if (gwait >= 0) bar_wait(P, gwait, ti); },
            [&]() {
                fold_swiglu(P, S, xbar);
                if (is_ctl_lane0()) trace_stamp(P, ti, 3);
            },
            [&](int) {},
            [&](int c, int b0, int nb, uint16_t *buf) {
                stage_bf16_chunk(P.actm + col0, P.actm_lo + col0, P.Fp, width, c, b0, nb, buf);
            },
            [&](int b, int r, float y0, float y1) {
                st_dev(part + (size_t)b * P.Hp + r, y0);
                st_dev(part + (size_t)b * P.Hp + r + 1, y1);
            },
            P.KTc, (size_t)P.down_rg * P.KTc);
    } else if (P.E > 1) {
        moe_down(P, S, l, ti);
    } else {
        const int j = blockIdx.x / P.Rc, part = blockIdx.x % P.Rc;
        if (j < P.Sc) {
            int a0, a1;
            split_range(P.down_rg, P.Rc, part, a0, a1);
            const int kw = P.KTc * kTileK, c0 = j * kw, nreal = max(0, min(kw, P.F - c0));
            weight_phase<false>(
                P, S, Wd + (size_t)j * P.down_rg * P.KTc * kTileBytes, P.KTc, a0, a1 - a0,
                [&]() {}, [&]() {},
                [&](int b) {
                    // block j of the SwiGLU output as tagged words, gathered
                    // by the control wave (its loads are not queued behind
                    // the weight ring); padding columns are zero.  With
                    // P.multi the first call gathers every sequence's block
                    // (block of sequence bb at a + bb kw).
                    if (b == 0 && is_ctl_lane0()) trace_stamp(P, ti, 1);
                    if (P.multi) {
                        if (b > 0) return;
                        if ((kl_tid() >> 6) == kCtlWave)
                            ll_gather<kDownGather>(
                                P, P.B * nreal, ll_tag(P, l), kl_tid() & 63, 64,
                                [&](int i) {
                                    const int bb = i / nreal;
                                    return P.m_ll + (size_t)bb * P.Fp + c0 + (i - bb * nreal);
                                },
                                [&](int i, unsigned v) {
                                    const int bb = i / nreal;
                                    S.a[bb * kw + (i - bb * nreal)] = __uint_as_float(v);
                                });
                        for (int i = kl_tid(); i < P.B * (kw - nreal); i += kThreads) {
                            const int bb = i / (kw - nreal);
                            S.a[bb * kw + nreal + (i - bb * (kw - nreal))] = 0.f;
                        }
                    } else {
                        if ((kl_tid() >> 6) == kCtlWave)
                            ll_gather<kDownGather>(
                                P, nreal, ll_tag(P, l), kl_tid() & 63, 64,
                                [&](int i) { return P.m_ll + (size_t)b * P.Fp + c0 + i; },
                                [&](int i, unsigned v) { S.a[i] = __uint_as_float(v); });
                        for (int i = nreal + kl_tid(); i < kw; i += kThreads) S.a[i] = 0.f;
                    }
                    lds_barrier();
                    if (b == 0 && is_ctl_lane0()) {
                        trace_stamp(P, ti, 2);
                        trace_stamp(P, ti, 3);
                    }
                },
                [&](int, int, int, uint16_t *) {}, epi, 0, 0, NoGroupDone(), kw);
        }
    }
    if (garrive >= 0) bar_arrive(P, garrive, ti);
}

// The final residual stream -> hidden_out (fp32).
template <bool PS>
__device__ __forceinline__ void copy_hidden(const StepParams &P) {
    for (int idx = kl_tid(); idx < P.B * P.H; idx += kThreads) {
        const int b = idx / P.H;
        const float x = from_fix((long long)ld_dev_u64(P.xf + (size_t)b * P.Hp + idx % P.H));
        P.hidden_out[idx] = ok_of<PS>(P, b) ? x : __builtin_nanf("");
    }
}

// Classifier block (Sec. 2): final RMSNorm + LM head -> fp32 logits.
template <bool BAT>
__device__ __forceinline__ void phase_head(KArg ka, int gwait, int ti) {
    const StepParams P = load_params(ka);
    const Lds S = lds_layout(kl_smem, P);
    const RgRange R = own_rgs(P.head_rg, P);
    const int V = P.V;
    // greedy sampling: this workgroup's best key per sequence (LDS atomics),
    // then one device-scope atomic per sequence into P.amax
    unsigned long long *best = amax_slots(P);
    const bool sample = P.amax != nullptr;
    if (sample && kl_tid() < kGemmBatch) best[kl_tid()] = 0ull;   // (staging barriers follow)
    auto flush = [&](int b0, int nb) {
        if (!sample) return;
        __syncthreads();
        const int t = kl_tid();
        if (t < nb) {
            const unsigned long long k = best[t];
            if (k) __hip_atomic_fetch_max(P.amax + b0 + t, k, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
            best[t] = 0ull;
        }
        __syncthreads();
    };
    weight_phase<BAT>(
        P, S, reinterpret_cast<const uint8_t *>(P.lm_head), P.Hp / kTileK, R.first, R.count,
        [&]() {
            if (gwait >= 0) bar_wait(P, gwait, ti);
            if (!BAT && blockIdx.x == 0 && P.hidden_out) copy_hidden<!BAT>(P);
        },
        [&]() {
            // (folds the last down projection's partials, x: xf2 -> xf), and
            // the sequences' RMSNorm scales for the epilogue
            norm_batched(P, S, P.final_norm, P.xf2, P.xf, P.KSd);
            norm_wait(P, 2 * P.L, 0, (P.Hp + kGemmChunkK - 1) / kGemmChunkK);
            __syncthreads();
            rms_table(P, S);
            if (is_ctl_lane0()) trace_stamp(P, ti, 3);
            if (blockIdx.x == 0 && P.hidden_out) copy_hidden<!BAT>(P);
        },
        [&](int b) {
            if (P.multi) {
                if (b == 0)
                    stage_rms_multi(P.xf, P.Hp, P.final_norm, P.H, P.Hp, P.B, S.a, P.Hp, S.sm,
                                    NoExtra(), NoExtra(), 0);
            } else {
                stage_rms_deferred(P.xf + (size_t)b * P.Hp, P.final_norm, P.H, P.Hp, S.a, S.sm);
            }
            if (b == 0 && is_ctl_lane0()) trace_stamp(P, ti, 3);
        },
        [&](int c, int b0, int nb, uint16_t *buf) { stage_act_chunk(P, c, b0, nb, buf); },
        [&](int b, int r, float y0, float y1) {
            // the deferred RMSNorm scale
            const float rs = !BAT ? rms_scale(seq_sm(P, S, b), P.H, P.eps) : rms_of(P, S, b);
            y0 *= rs;
            y1 *= rs;
            const bool ok = ok_of<!BAT>(P, b);
            if (!ok) y0 = y1 = __builtin_nanf("");
            float *lg = P.logits + (size_t)b * V;
            if (r < V) lg[r] = y0;
            if (r + 1 < V) lg[r + 1] = y1;
            if (sample && ok) {
                unsigned long long k = (r < V) ? argmax_key(y0, r) : 0ull;
                if (r + 1 < V) k = max(k, argmax_key(y1, r + 1));
                __hip_atomic_fetch_max(best + (BAT ? b % kGemmBatch : b), k, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        },
        0, 0, [&](int b0, int nb) { flush(b0, nb); }, P.Hp);
    if (!BAT) flush(0, P.B);
    // the step's last phase: the next step's tags (every workgroup of every
    // launch of this step read the epoch at its start)
    if (blockIdx.x == 0 && kl_tid() == 0)
        __hip_atomic_store(P.epoch_ptr, ll_next_epoch(*launch_epoch(P), P.L), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    if (is_ctl_lane0()) trace_stamp(P, ti, 0);
}

// ---------------------------------------------------------------- kernels

// Runs the phases selected by 'phases' for layers [l0, l1) in order:
// embed, (qkv, attn, oproj, gateup, down) per layer, head.  Grid barrier k is
// the k-th arrival of the launch; a phase that needs the residual stream waits
// on the latest one, and an arriving phase arrives only if a later phase of
// the same launch waits (a launch boundary already orders the rest).
template <int D, int G, bool BAT>
__global__ __launch_bounds__(kThreads) void kl_step_kernel(StepParams P, int l0, int l1,
                                                          int phases) {
    (void)P;   // read through the kernel-argument segment (see load_params)
    const KArg ka = kernarg_address();
    const bool has_qkv = phases & kPhQkv, has_gu = phases & kPhGateUp, has_head = phases & kPhHead;
    const int nlay = (phases & kPhLayer) ? l1 - l0 : 0;
    // batched steps add grid barriers of their own: after the q/k/v product
    // (its fold), in the SwiGLU fold, and before a merge of several attention
    // chunks (their RMSNorm steps hand over through slice counters instead)
    constexpr bool batched = BAT;
    bar_init(load_params(ka));
    int na = 0, ti = 0;   // grid arrivals so far; phase index (for the trace)
    auto gw = [&]() { return na - 1; };                 // barrier to wait on (-1: none)
    auto ga = [&](bool waited_later) { return waited_later ? na++ : -1; };
    auto xb = [&]() { return batched ? na++ : -1; };    // the phase's own barrier
    const bool has_attn = phases & kPhAttn, has_op = phases & kPhOproj;
    const bool has_down = phases & kPhDown;
    if (phases & kPhEmbed) {
        phase_embed(ka, -1, ga((has_qkv && nlay > 0) || has_head), ti++);
    }
    for (int l = l0; l < l1; ++l) {
        // batched steps: attn -> oproj and gateup -> down are grid barriers
        // too (full-K products with one writer per output)
        if (phases & kPhQkv) {
            const int w = gw(), q = xb();
            phase_qkv<BAT>(ka, l, w, q, ti++);
        }
        if (phases & kPhAttn) phase_attn<D, G, BAT>(ka, l, BAT ? ga(has_op) : -1, ti++);
        if (phases & kPhOproj) {
            // (batched, several attention chunks: the merge step's own barrier)
            const int w = BAT && has_attn ? gw() : -1;
            const int m = BAT && load_params(ka).C > 1 ? na++ : -1, a = ga(has_gu);
            phase_oproj<D, G, BAT>(ka, l, w, m, a, ti++);
        }
        if (phases & kPhGateUp) {
            const int w = gw(), a = BAT ? ga(has_down) : -1;
            phase_gateup<BAT>(ka, l, w, a, ti++);
        }
        if (phases & kPhDown) {
            // (batched: the SwiGLU fold of the gate/up partials ends with a
            // grid barrier of its own)
            const int w = BAT && has_gu ? gw() : -1, x = xb();
            phase_down<BAT>(ka, l, w, x, ga((has_qkv && l + 1 < l1) || has_head), ti++);
        }
    }
    if (has_head) {
        phase_head<BAT>(ka, gw(), ti++);
    }
}

}  // namespace kl
