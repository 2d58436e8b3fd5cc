// moe_decode.hip -- the expert FFN for small token counts (decode: at most 16
// tokens per expert), streamed from HBM.
//
// Each workgroup owns one 16-feature tile of one active expert; wave w of its
// kSplit waves takes the K tiles w, w + kSplit, w + 2 kSplit, ... (so at each
// step the waves together read kSplit x unroll consecutive 1 KiB tiles of
// the slab), and wave 0 adds the partial fragments in wave order
// (deterministic) before the epilogue.  Splitting K keeps enough loads in
// flight when few experts are active (one expert of an expert-parallel share
// has only 672 gate/up and 384 down tiles).  The weight tile is the A operand of v_mfma_f32_16x16x32_bf16
// and the (at most 16) tokens of the expert are the B operand, so the matrix
// cores do the dot products and the reduction over K; the kernel is a pure
// 16-byte-per-lane stream of the packed weights (every wave-wide load is 1 KiB
// contiguous).  Lanes whose token column is unused feed zeros.
//
// gateup_kernel: G = x W1, U = x V1 for the 16 features, then
//                H = bf16(silu(G) * U)          (paper Table tab:vars (e): w1, v1)
// down_kernel:   O = H W2 for 16 output features, fp32
//
// Output fragment of the MFMA: lane l holds rows 4*(l/16)+r (r = 0..3) of
// column l%16, i.e. four consecutive features of token slot l%16.
#include "moe_common.h"

namespace moe {

constexpr int kSplit = 8;    // waves per workgroup (K split)
// K tiles per wave per step (loads in flight per slab and wave).  Measured
// on the decode step: gate/up is flat over 4..8; down is fastest at 6 (8 and
// 12 hold more registers for no gain, 2..4 keep too few loads in flight).
constexpr int kUnrollGU = 8;
constexpr int kUnrollDN = 6;

// partial fragments of waves 1.. through LDS; wave 0 adds them in wave order
__device__ inline void reduce_waves(f32x4_t& v, f32x4_t* s, int w, int lane)
{
    if (w > 0) s[(w - 1) * 64 + lane] = v;
    __syncthreads();
    if (w == 0)
        for (int i = 0; i + 1 < kSplit; ++i) v += s[i * 64 + lane];
}

__device__ inline u32x4_t ld16(const void* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}

__device__ inline u32x4_t ld16_cached(const void* p)
{
    return *reinterpret_cast<const u32x4_t*>(p);
}

__global__ __launch_bounds__(64 * kSplit) void gateup_kernel(DecodeArgs a)
{
    __shared__ f32x4_t s_red[2 * (kSplit - 1) * 64];
    const int n_ftiles = a.f / kTileRows;
    const int slot = blockIdx.x / n_ftiles;
    const int p = blockIdx.x % n_ftiles;
    if (slot >= a.active[0]) return;
    const int e = a.active[1 + slot];
    const int m = a.counts[e];
    const int row0 = a.offsets[e];
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int j = lane & 15;     // token slot (B column)
    const int g = lane >> 4;     // K group of 8

    const int KT = a.d / kTileK;
    const uint8_t* base = a.experts + (uint64_t)(e - a.e_begin) * a.expert_bytes;
    const uint8_t* pg = base + tile_offset(2 * p, 0, KT) + lane * 16;
    const uint8_t* pu = base + tile_offset(2 * p + 1, 0, KT) + lane * 16;
    const bool has_tok = j < m;
    const uint16_t* px = a.x + (has_tok ? (int64_t)a.row_token[row0 + j] * a.d : 0) + g * 8;

    f32x4_t acc_g = {0.f, 0.f, 0.f, 0.f};
    f32x4_t acc_u = {0.f, 0.f, 0.f, 0.f};
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    // wave w takes K tiles w, w + kSplit, ...: per step the workgroup's waves
    // read kSplit * kUnrollGU consecutive tiles of each slab
    int kt = 0;
    for (; kt + kSplit * kUnrollGU <= KT; kt += kSplit * kUnrollGU) {
        u32x4_t wg[kUnrollGU], wu[kUnrollGU], xb[kUnrollGU];
#pragma unroll
        for (int u = 0; u < kUnrollGU; ++u) {
            wg[u] = ld16(pg + (int64_t)(kt + w + kSplit * u) * kTileBytes);
            wu[u] = ld16(pu + (int64_t)(kt + w + kSplit * u) * kTileBytes);
        }
#pragma unroll
        for (int u = 0; u < kUnrollGU; ++u)
            xb[u] = has_tok ? ld16_cached(px + (kt + w + kSplit * u) * kTileK) : zero;
#pragma unroll
        for (int u = 0; u < kUnrollGU; ++u) {
            acc_g = mfma16x16x32(wg[u], xb[u], acc_g);
            acc_u = mfma16x16x32(wu[u], xb[u], acc_u);
        }
    }
    for (kt += w; kt < KT; kt += kSplit) {
        const u32x4_t wg = ld16(pg + (int64_t)kt * kTileBytes), wu = ld16(pu + (int64_t)kt * kTileBytes);
        const u32x4_t xb = has_tok ? ld16_cached(px + kt * kTileK) : zero;
        acc_g = mfma16x16x32(wg, xb, acc_g);
        acc_u = mfma16x16x32(wu, xb, acc_u);
    }
    reduce_waves(acc_g, s_red, w, lane);
    reduce_waves(acc_u, s_red + (kSplit - 1) * 64, w, lane);
    if (w != 0) return;
    if (has_tok) {
        uint32_t h01 = (uint32_t)f32_to_bf16(silu_mul(acc_g[0], acc_u[0])) |
                       ((uint32_t)f32_to_bf16(silu_mul(acc_g[1], acc_u[1])) << 16);
        uint32_t h23 = (uint32_t)f32_to_bf16(silu_mul(acc_g[2], acc_u[2])) |
                       ((uint32_t)f32_to_bf16(silu_mul(acc_g[3], acc_u[3])) << 16);
        uint16_t* ph = a.H + (int64_t)(row0 + j) * a.f + p * kTileRows + g * 4;
        *reinterpret_cast<uint2*>(ph) = make_uint2(h01, h23);
    }
}

__global__ __launch_bounds__(64 * kSplit) void down_kernel(DecodeArgs a)
{
    __shared__ f32x4_t s_red[(kSplit - 1) * 64];
    const int n_otiles = a.d / kTileRows;
    const int slot = blockIdx.x / n_otiles;
    const int q = blockIdx.x % n_otiles;
    if (slot >= a.active[0]) return;
    const int e = a.active[1 + slot];
    const int m = a.counts[e];
    const int row0 = a.offsets[e];
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int j = lane & 15;
    const int g = lane >> 4;

    const int KT = a.f / kTileK;
    const uint8_t* base = a.experts + (uint64_t)(e - a.e_begin) * a.expert_bytes + a.gu_bytes;
    const uint8_t* pw = base + tile_offset(q, 0, KT) + lane * 16;
    const bool has_tok = j < m;
    const uint16_t* ph = a.H + (has_tok ? (int64_t)(row0 + j) * a.f : 0) + g * 8;

    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    int kt = 0;
    for (; kt + kSplit * kUnrollDN <= KT; kt += kSplit * kUnrollDN) {
        u32x4_t wv[kUnrollDN], hb[kUnrollDN];
#pragma unroll
        for (int u = 0; u < kUnrollDN; ++u)
            wv[u] = ld16(pw + (int64_t)(kt + w + kSplit * u) * kTileBytes);
#pragma unroll
        for (int u = 0; u < kUnrollDN; ++u)
            hb[u] = has_tok ? ld16_cached(ph + (kt + w + kSplit * u) * kTileK) : zero;
#pragma unroll
        for (int u = 0; u < kUnrollDN; ++u) acc = mfma16x16x32(wv[u], hb[u], acc);
    }
    for (kt += w; kt < KT; kt += kSplit) {
        const u32x4_t wv = ld16(pw + (int64_t)kt * kTileBytes);
        const u32x4_t hb = has_tok ? ld16_cached(ph + kt * kTileK) : zero;
        acc = mfma16x16x32(wv, hb, acc);
    }
    reduce_waves(acc, s_red, w, lane);
    if (w != 0) return;
    if (has_tok) {
        float* po = a.O + (int64_t)(row0 + j) * a.d + q * kTileRows + g * 4;
        *reinterpret_cast<float4*>(po) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
}

}  // namespace moe

extern "C" hipError_t moe_launch_decode_gateup(const moe::DecodeArgs* a, int n_slots,
                                               hipStream_t s)
{
    const int blocks = n_slots * (a->f / moe::kTileRows);
    hipLaunchKernelGGL(moe::gateup_kernel, dim3(blocks), dim3(64 * moe::kSplit), 0, s, *a);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_decode_down(const moe::DecodeArgs* a, int n_slots, hipStream_t s)
{
    const int blocks = n_slots * (a->d / moe::kTileRows);
    hipLaunchKernelGGL(moe::down_kernel, dim3(blocks), dim3(64 * moe::kSplit), 0, s, *a);
    return hipGetLastError();
}
