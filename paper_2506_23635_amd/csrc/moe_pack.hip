// moe_pack.hip -- expert prestacking (paper Sec. 4.1): one-time repack of an
// expert's boundary-layout matrices into the arena's fragment-tiled layout
// (described in moe_common.h).
//
// A source matrix is row-major [K][N] (K = reduction dim, N = output
// features): gate/up are [d][f], down is [f][d].  The packed matrix is
// feature-major with K contiguous, so the repack is a transpose, done through
// LDS in 64 x 64 blocks so that both the reads and the writes are coalesced.
#include "moe_common.h"

namespace moe {

// One block repacks src[k0:k0+64][n0:n0+64].  Feature n lands in row tile
// (n'/16)*rt_mul + rt_add of the destination, which has KT = K/32 K tiles;
// n' = n, or rope_row(n) for the features below perm_rows.
__global__ __launch_bounds__(256) void pack_kernel(const uint16_t* __restrict__ src, int K, int N,
                                                   uint8_t* __restrict__ dst, int rt_mul,
                                                   int rt_add, int perm_hd, int perm_rows)
{
    __shared__ uint16_t tile[64][64 + 2];
    const int n0 = blockIdx.x * 64;
    const int k0 = blockIdx.y * 64;
    const int t = threadIdx.x;
    // load: 64 rows x 8 granules of 8 bf16, two granules per thread
    for (int c = t; c < 512; c += 256) {
        int r = c >> 3, g = c & 7;
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(src + (int64_t)(k0 + r) * N + n0 + g * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            tile[r][g * 8 + 2 * e] = (uint16_t)(v[e] & 0xFFFFu);
            tile[r][g * 8 + 2 * e + 1] = (uint16_t)(v[e] >> 16);
        }
    }
    __syncthreads();
    // store: 64 features x 8 K-granules; granule = (feature n, K group kg)
    const uint64_t KT = (uint64_t)K / kTileK;
    for (int c = t; c < 512; c += 256) {
        int nl = c & 63;        // feature within block (fastest: contiguous lanes)
        int kg = c >> 6;        // 8-wide K group within the 64-K block (0..7)
        int n = n0 + nl;
        if (n < perm_rows) n = rope_row(n, perm_hd);
        int kk = kg * 8;        // K offset within block
        u32x4_t w;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            w[e] = (uint32_t)tile[kk + 2 * e][nl] | ((uint32_t)tile[kk + 2 * e + 1][nl] << 16);
        uint64_t rt = (uint64_t)(n / kTileRows) * rt_mul + rt_add;
        uint64_t kt = (uint64_t)(k0 + kk) / kTileK;
        int lane = ((kk % kTileK) / 8) * 16 + (n % kTileRows);
        uint8_t* p = dst + tile_offset(rt, kt, KT) + (uint64_t)lane * 16;
        *reinterpret_cast<u32x4_t*>(p) = w;
    }
}

}  // namespace moe

extern "C" hipError_t moe_launch_pack_perm(const uint16_t* src, int K, int N, void* dst,
                                           int rt_mul, int rt_add, int perm_hd, int perm_rows,
                                           hipStream_t s)
{
    dim3 grid(N / 64, K / 64);
    hipLaunchKernelGGL(moe::pack_kernel, grid, dim3(256), 0, s, src, K, N, (uint8_t*)dst, rt_mul,
                       rt_add, perm_hd, perm_rows);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_pack(const uint16_t* src, int K, int N, void* dst, int rt_mul,
                                      int rt_add, hipStream_t s)
{
    return moe_launch_pack_perm(src, K, N, dst, rt_mul, rt_add, 0, 0, s);
}

// The same repack on the host, for weights that arrive in host memory.
extern "C" void moe_pack_host_perm(const uint16_t* src, int K, int N, uint8_t* dst, int rt_mul,
                                   int rt_add, int perm_hd, int perm_rows)
{
    const uint64_t KT = (uint64_t)K / moe::kTileK;
    for (int n0 = 0; n0 < N; ++n0) {
        const int n = n0 < perm_rows ? moe::rope_row(n0, perm_hd) : n0;
        const uint64_t rt = (uint64_t)(n / moe::kTileRows) * rt_mul + rt_add;
        for (int k0 = 0; k0 < K; k0 += 8) {
            const uint64_t kt = (uint64_t)k0 / moe::kTileK;
            const int lane = ((k0 % moe::kTileK) / 8) * 16 + (n % moe::kTileRows);
            uint16_t* p = reinterpret_cast<uint16_t*>(dst + moe::tile_offset(rt, kt, KT) + lane * 16);
            for (int i = 0; i < 8; ++i) p[i] = src[(size_t)(k0 + i) * N + n0];
        }
    }
}

extern "C" void moe_pack_host(const uint16_t* src, int K, int N, uint8_t* dst, int rt_mul,
                              int rt_add)
{
    moe_pack_host_perm(src, K, N, dst, rt_mul, rt_add, 0, 0);
}
