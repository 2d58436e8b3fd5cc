// Device build of the seeded input generator (definition in philox_gen.h).
// Writes synthetic tensors straight into HBM so that multi-GB weight sets
// never cross PCIe; the bits equal the host build's.
#include <hip/hip_runtime.h>
#include "philox_gen.h"

__global__ __launch_bounds__(256) void moe_gen_bf16_kernel(uint32_t seed, uint32_t stream,
                                                           uint64_t start, int64_t n, double c,
                                                           uint16_t* __restrict__ out)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += step)
        out[i] = moe_gen_bf16(seed, stream, start + (uint64_t)i, c);
}

__global__ __launch_bounds__(256) void moe_gen_f32_kernel(uint32_t seed, uint32_t stream,
                                                          uint64_t start, int64_t n, double c,
                                                          float* __restrict__ out)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += step)
        out[i] = moe_gen_f32(seed, stream, start + (uint64_t)i, c);
}

static int grid_for(int64_t n)
{
    int64_t g = (n + 255) / 256;
    if (g > 256 * 64) g = 256 * 64;
    if (g < 1) g = 1;
    return (int)g;
}

extern "C" int moe_gen_fill_bf16_device(uint32_t seed, uint32_t stream, uint64_t start,
                                        int64_t n, double c, void* dst, void* stream_handle)
{
    if (n < 0 || (n > 0 && dst == nullptr)) return -1;
    if (n == 0) return 0;
    hipStream_t s = (hipStream_t)stream_handle;
    hipLaunchKernelGGL(moe_gen_bf16_kernel, dim3(grid_for(n)), dim3(256), 0, s, seed, stream,
                       start, n, c, (uint16_t*)dst);
    return hipGetLastError() == hipSuccess ? 0 : -6;
}

extern "C" int moe_gen_fill_f32_device(uint32_t seed, uint32_t stream, uint64_t start,
                                       int64_t n, double c, void* dst, void* stream_handle)
{
    if (n < 0 || (n > 0 && dst == nullptr)) return -1;
    if (n == 0) return 0;
    hipStream_t s = (hipStream_t)stream_handle;
    hipLaunchKernelGGL(moe_gen_f32_kernel, dim3(grid_for(n)), dim3(256), 0, s, seed, stream,
                       start, n, c, (float*)dst);
    return hipGetLastError() == hipSuccess ? 0 : -6;
}
