// moe_diag.hip -- diagnostics beside the layer: a plain streaming read of a
// device buffer, the achievable HBM read rate that the layer's weight
// streams are compared with (the spec peak is 8 TB/s); and the hardware
// fp32 -> bf16 conversion of the grouped GEMM's gate/up epilogue, applied to
// a caller's array so that it can be checked against round-to-nearest-even
// on every fp32 pattern.
//
// The streaming read:
// Each workgroup reads one contiguous chunk of the buffer: per iteration
// its 256 lanes load 8 x 4 KiB of consecutive 16-byte words (1 KiB per
// wave-load, nontemporal, eight loads in flight per lane), and XOR them; the
// workgroup's XOR goes to its own 16 bytes of out (no atomics, no shared
// address), so no load is dead.
#include "moe_common.h"

#include "../../include/moe.h"

namespace moe {

constexpr int kDiagThreads = 256;
constexpr int kDiagUnroll = 8;

__global__ __launch_bounds__(kDiagThreads) void stream_read_kernel(const u32x4_t* __restrict__ p,
                                                                   uint64_t n_words, uint32_t* out)
{
    const uint64_t per_wg = (n_words + gridDim.x - 1) / gridDim.x;
    const uint64_t w0 = (uint64_t)blockIdx.x * per_wg;
    const uint64_t w1 = w0 + per_wg < n_words ? w0 + per_wg : n_words;
    uint64_t i = w0 + threadIdx.x;
    u32x4_t acc = {0u, 0u, 0u, 0u};
    for (; i + (kDiagUnroll - 1) * kDiagThreads < w1; i += kDiagUnroll * kDiagThreads) {
        u32x4_t v[kDiagUnroll];
#pragma unroll
        for (int u = 0; u < kDiagUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * kDiagThreads);
#pragma unroll
        for (int u = 0; u < kDiagUnroll; ++u) acc ^= v[u];
    }
    for (; i < w1; i += kDiagThreads) acc ^= __builtin_nontemporal_load(p + i);
#pragma unroll
    for (int c = 0; c < 4; ++c)
        for (int off = kWave / 2; off >= 1; off >>= 1) acc[c] ^= __shfl_xor(acc[c], off, kWave);
    __shared__ u32x4_t s_acc[kDiagThreads / kWave];
    const int wv = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) s_acc[wv] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        u32x4_t r = s_acc[0];
        for (int k = 1; k < kDiagThreads / kWave; ++k) r ^= s_acc[k];
        reinterpret_cast<u32x4_t*>(out)[blockIdx.x] = r;
    }
}

// y[i] = bf16(x[i]) by cvt_pk_bf16, two elements per thread, grid-stride
__global__ __launch_bounds__(kDiagThreads) void bf16_convert_kernel(const float2* __restrict__ x,
                                                                    uint32_t* __restrict__ y,
                                                                    uint64_t n_pairs)
{
    for (uint64_t i = (uint64_t)blockIdx.x * kDiagThreads + threadIdx.x; i < n_pairs;
         i += (uint64_t)gridDim.x * kDiagThreads) {
        const float2 v = x[i];
        y[i] = cvt_pk_bf16(v.x, v.y);
    }
}

}  // namespace moe

extern "C" moe_status moe_diag_bf16(const float* src, uint16_t* dst, uint64_t n, moe_stream_t stream)
{
    if (!src || !dst || ((uintptr_t)src & 7) || ((uintptr_t)dst & 3) || n % 2) return MOE_E_ARG;
    if (n == 0) return MOE_OK;
    const uint64_t n_pairs = n / 2;
    const uint64_t want = (n_pairs + moe::kDiagThreads - 1) / moe::kDiagThreads;
    const int grid = (int)(want < 8192 ? want : 8192);
    hipLaunchKernelGGL(moe::bf16_convert_kernel, dim3(grid), dim3(moe::kDiagThreads), 0,
                       static_cast<hipStream_t>(stream), reinterpret_cast<const float2*>(src),
                       reinterpret_cast<uint32_t*>(dst), n_pairs);
    return hipGetLastError() == hipSuccess ? MOE_OK : MOE_E_HIP;
}

extern "C" moe_status moe_diag_stream_read(const void* src, uint64_t bytes, uint32_t* out,
                                           moe_stream_t stream)
{
    if (!src || !out || ((uintptr_t)src & 15) || ((uintptr_t)out & 15) || bytes % 16)
        return MOE_E_ARG;
    if (bytes == 0) return MOE_OK;
    // at most two workgroups of 256 threads per CU (256 CUs), at least 16 KiB
    // each: measured, a few long contiguous chunks read faster than many short
    // ones (7.2 TB/s at 512 workgroups, 6.8 at 2048, 6.5 at 4096 for 4 GiB)
    const uint64_t n_words = bytes / 16;
    const int grid = (int)(n_words / 1024 < MOE_DIAG_MAX_WG ? (n_words / 1024 > 0 ? n_words / 1024 : 1)
                                                           : MOE_DIAG_MAX_WG);
    hipLaunchKernelGGL(moe::stream_read_kernel, dim3(grid), dim3(moe::kDiagThreads), 0,
                       static_cast<hipStream_t>(stream), static_cast<const moe::u32x4_t*>(src),
                       n_words, out);
    return hipGetLastError() == hipSuccess ? MOE_OK : MOE_E_HIP;
}
