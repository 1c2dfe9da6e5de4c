// Host-side entry points of the device code: the step-kernel selector and
// launchers, and the load-time packing kernels.

#include <algorithm>
#include <mutex>
#include <unordered_map>

#include "kl_step_impl.h"

namespace kl {

// The scratch of the entry point that allocates nothing
// (kl_decode_step_noalloc): a file-scope device array, one copy per device
// that loads this library, kept until the process ends.  In host code its name
// stands for no device address: host code uses only the address
// static_scratch_address returns.
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

hipError_t static_scratch_address(int device, uint8_t **out) {
    static std::mutex mu;
    static std::unordered_map<int, uint8_t *> addr;   // device -> its copy's address
    std::lock_guard<std::mutex> lock(mu);
    const auto it = addr.find(device);
    if (it != addr.end()) {
        *out = it->second;
        return hipSuccess;
    }
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[device] = static_cast<uint8_t *>(p);
    *out = static_cast<uint8_t *>(p);
    return hipSuccess;
}

__global__ void kl_zero_kernel(u32x4 *p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = u32x4{0u, 0u, 0u, 0u};
}

hipError_t launch_zero(void *p, size_t bytes, hipStream_t stream) {
    const size_t n = bytes / 16;
    if (n == 0) return hipSuccess;
    const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(kl_zero_kernel, dim3(blocks), dim3(256), 0, stream,
                       reinterpret_cast<u32x4 *>(p), n);
    return hipGetLastError();
}

// Read stream: every 16-byte chunk of the buffer is loaded once with the
// step kernel's load (non-temporal, 16 B per lane), 16 loads in flight per
// lane; in round r, lane t of the grid's T lanes loads chunks (16 r + j) T + t,
// j < 16, so a wave reads 1 KiB runs.  The loaded words are folded into one
// value that is stored only if it equals a constant the data never produce
// (the loads cannot be dropped, and nothing is written).
__global__ void __launch_bounds__(512) kl_read_stream_kernel(const u32x4 *__restrict__ p,
                                                             size_t n, uint32_t *out) {
    const size_t T = (size_t)gridDim.x * blockDim.x;
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t acc = 0;
    for (size_t base = 0; base < n; base += 16 * T) {
        u32x4 v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const size_t i = base + j * T + t;
            v[j] = i < n ? ld_stream_16B(p + i) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) acc ^= v[j][0] ^ v[j][1] ^ v[j][2] ^ v[j][3];
    }
    if (acc == 0x9E3779B9u) out[0] = acc;
}

hipError_t launch_read_stream(const void *p, size_t bytes, int workgroups, uint32_t *out,
                              hipStream_t stream) {
    hipLaunchKernelGGL(kl_read_stream_kernel, dim3(workgroups), dim3(512), 0, stream,
                       reinterpret_cast<const u32x4 *>(p), bytes / 16, out);
    return hipGetLastError();
}

// The instance for a model's head_dim, query heads per KV head (the host has
// validated both) and the batch regime (the matrix cores when p.batched);
// the instances are compiled in separate translation units (kl_step_*.hip).
StepKernel step_kernel_for(int d, int group, bool batched) {
    if (d == 64) return batched ? step_kernel_d64_batched(group) : step_kernel_d64(group);
    if (d == 128) return batched ? step_kernel_d128_batched(group) : step_kernel_d128(group);
    return nullptr;
}

// Repack row-major bf16 matrices (row stride ld elements) into 8x64 tiles of
// their first K columns, one 16-byte chunk per thread (pack_chunk: the row
// map gives each packed row's source and row, columns >= K are zero).
__global__ void kl_pack_rows_kernel(uint16_t *__restrict__ dst, int n_rg, int KT, int K, int ld,
                                    const int32_t *__restrict__ rowmap,
                                    const uint16_t *__restrict__ s0,
                                    const uint16_t *__restrict__ s1,
                                    const uint16_t *__restrict__ s2) {
    const size_t chunks = (size_t)n_rg * KT * 64;
    const uint16_t *const src[3] = {s0, s1, s2};
    for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < chunks;
         idx += (size_t)gridDim.x * blockDim.x) {
        uint32_t w[4];
        pack_chunk(idx, KT, K, ld, rowmap, src, w);
        reinterpret_cast<u32x4 *>(dst)[idx] = u32x4{w[0], w[1], w[2], w[3]};
    }
}

__global__ void kl_emit_tokens_kernel(int32_t *tokens, const unsigned long long *keys, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) tokens[i] = key_token(keys[i]);
}

hipError_t launch_emit_tokens(int32_t *tokens, const unsigned long long *keys, int n,
                              hipStream_t stream) {
    hipLaunchKernelGGL(kl_emit_tokens_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, tokens,
                       keys, n);
    return hipGetLastError();
}

__global__ void kl_pack_bias_kernel(float *dst, int rows, const int32_t *__restrict__ rowmap,
                                    const uint16_t *b0, const uint16_t *b1, const uint16_t *b2) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    const uint16_t *const src[3] = {b0, b1, b2};
    dst[r] = pack_bias_row(r, rowmap, src);
}

hipError_t launch_pack_bias(float *dst, int rows, const int32_t *rowmap, const uint16_t *bq,
                            const uint16_t *bk, const uint16_t *bv, hipStream_t stream) {
    hipLaunchKernelGGL(kl_pack_bias_kernel, dim3((rows + 255) / 256), dim3(256), 0, stream, dst,
                       rows, rowmap, bq, bk, bv);
    return hipGetLastError();
}

__global__ void kl_gain_to_f32_kernel(float *dst, const uint16_t *src, int n, int npad) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < npad; i += gridDim.x * blockDim.x)
        dst[i] = (i < n) ? bf2f(src[i]) : 0.f;
}

// ---------------------------------------------------------------- launchers

hipError_t step_kernel_setup(int d, int group, int lds_bytes, int *max_blocks_per_cu) {
    *max_blocks_per_cu = 1 << 30;
    for (int bat = 0; bat < 2; ++bat) {
        const StepKernel k = step_kernel_for(d, group, bat != 0);
        if (!k) return hipErrorInvalidValue;
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
        if (e != hipSuccess) return e;
        int n = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, kThreads, lds_bytes);
        if (e != hipSuccess) return e;
        *max_blocks_per_cu = std::min(*max_blocks_per_cu, n);
    }
    return hipSuccess;
}

hipError_t launch_step(const StepParams &p, int first_layer, int last_layer, int phases,
                       bool cooperative, int lds_bytes, hipStream_t stream) {
    const StepKernel k = step_kernel_for(p.d, p.group, p.batched != 0);
    if (!k) return hipErrorInvalidValue;
    StepParams pc = p;
    if (cooperative) {
        void *args[] = {&pc, &first_layer, &last_layer, &phases};
        return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(k), dim3(p.nwg),
                                          dim3(kThreads), args, lds_bytes, stream);
    }
    hipLaunchKernelGGL(k, dim3(p.nwg), dim3(kThreads), lds_bytes, stream, pc, first_layer,
                       last_layer, phases);
    return hipGetLastError();
}

hipError_t add_step_node(hipGraph_t g, hipGraphNode_t *node, const hipGraphNode_t *dep,
                         const StepParams &p, int first_layer, int last_layer, int phases,
                         bool cooperative, int lds_bytes) {
    const StepKernel k = step_kernel_for(p.d, p.group, p.batched != 0);
    if (!k) return hipErrorInvalidValue;
    StepParams pc = p;   // (the node copies its arguments when it is added)
    void *args[] = {&pc, &first_layer, &last_layer, &phases};
    hipKernelNodeParams kp{};
    kp.func = reinterpret_cast<void *>(k);
    kp.gridDim = dim3(p.nwg);
    kp.blockDim = dim3(kThreads);
    kp.sharedMemBytes = (unsigned)lds_bytes;
    kp.kernelParams = args;
    hipError_t e = hipGraphAddKernelNode(node, g, dep, dep ? 1 : 0, &kp);
    if (e != hipSuccess || !cooperative) return e;
    hipKernelNodeAttrValue v{};
    v.cooperative = 1;
    return hipGraphKernelNodeSetAttribute(*node, hipKernelNodeAttributeCooperative, &v);
}

hipError_t launch_pack_rows(uint16_t *dst, int n_rg, int kt, int K, int ld, const int32_t *rowmap,
                            const uint16_t *src0, const uint16_t *src1, const uint16_t *src2,
                            hipStream_t stream) {
    const size_t chunks = (size_t)n_rg * kt * 64;
    const int blocks = (int)std::min<size_t>((chunks + 255) / 256, 65536);
    hipLaunchKernelGGL(kl_pack_rows_kernel, dim3(blocks), dim3(256), 0, stream, dst, n_rg, kt, K,
                       ld, rowmap, src0, src1, src2);
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
