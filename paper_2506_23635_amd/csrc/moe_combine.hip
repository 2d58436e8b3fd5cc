// moe_combine.hip -- the weighted sum of the selected experts' outputs back in
// token order (paper Sec. 2.2: after the router-selected experts finish, their
// outputs are combined by a weighted sum; Sec. 4.2: experts a token did not
// select contribute zero).
//
// y[t, n] = bf16( sum over slots j of t with a local expert: w[t,j] * O[row(t,j), n] )
// The slots are summed in slot order in fp32 by the one thread that owns the
// element, so the result is deterministic (no atomics).  With y32 set the
// unrounded fp32 sums are written instead (an expert-parallel share's partial
// for a later cross-device reduction).  With a residual the kernel instead
// writes x[t, n] = bf16(x[t, n] + y[t, n]) in place.
//
// The residual sum is one correct rounding although it is formed in fp32: two
// bf16 values whose exponents differ by at most 15 add exactly in fp32's 24
// bits; with a larger gap the smaller one is below 2^-15 of the larger, less
// than half a bf16 step, so both the exact sum and its fp32 rounding round
// to the larger value.
#include "moe_common.h"

namespace moe {

__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ O,
                                                      const int32_t* __restrict__ pair_row,
                                                      const float* __restrict__ topk_w, int T,
                                                      int d, int k, uint16_t* __restrict__ y,
                                                      float* __restrict__ y32,
                                                      uint16_t* __restrict__ x_residual)
{
    const int groups = d / 8;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (int64_t)T * groups) return;
    const int t = (int)(gid / groups);
    const int n = (int)(gid % groups) * 8;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
        const int r = pair_row[(int64_t)t * k + j];
        if (r < 0) continue;
        const float w = topk_w[(int64_t)t * k + j];
        const float4* po = reinterpret_cast<const float4*>(O + (int64_t)r * d + n);
        const float4 a = po[0], b = po[1];
        acc[0] = fmaf(w, a.x, acc[0]); acc[1] = fmaf(w, a.y, acc[1]);
        acc[2] = fmaf(w, a.z, acc[2]); acc[3] = fmaf(w, a.w, acc[3]);
        acc[4] = fmaf(w, b.x, acc[4]); acc[5] = fmaf(w, b.y, acc[5]);
        acc[6] = fmaf(w, b.z, acc[6]); acc[7] = fmaf(w, b.w, acc[7]);
    }
    u32x4_t out;
    if (x_residual) {
        u32x4_t xv = *reinterpret_cast<const u32x4_t*>(x_residual + (int64_t)t * d + n);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint32_t lo = 0, hi = 0;
            for (int h = 0; h < 2; ++h) {
                const uint16_t xb = (uint16_t)(xv[i] >> (16 * h));
                const uint16_t yb = f32_to_bf16(acc[2 * i + h]);
                (h ? hi : lo) = f32_to_bf16(bf16_to_f32(xb) + bf16_to_f32(yb));
            }
            out[i] = lo | (hi << 16);
        }
        *reinterpret_cast<u32x4_t*>(x_residual + (int64_t)t * d + n) = out;
    } else if (y32) {
        float4* py = reinterpret_cast<float4*>(y32 + (int64_t)t * d + n);
        py[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        py[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            out[i] = (uint32_t)f32_to_bf16(acc[2 * i]) |
                     ((uint32_t)f32_to_bf16(acc[2 * i + 1]) << 16);
        *reinterpret_cast<u32x4_t*>(y + (int64_t)t * d + n) = out;
    }
}

}  // namespace moe

extern "C" hipError_t moe_launch_combine(const float* O, const int32_t* pair_row,
                                         const float* topk_w, int T, int d, int k, uint16_t* y,
                                         float* y32, uint16_t* x_residual, hipStream_t s)
{
    int64_t total = (int64_t)T * (d / 8);
    int grid = (int)((total + 255) / 256);
    hipLaunchKernelGGL(moe::combine_kernel, dim3(grid), dim3(256), 0, s, O, pair_row, topk_w, T,
                       d, k, y, y32, x_residual);
    return hipGetLastError();
}
