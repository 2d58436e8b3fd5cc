// moe_prefill.hip -- the expert FFN for many tokens (prefill): a grouped GEMM
// on the bf16 matrix cores (v_mfma_f32_16x16x32_bf16).
//
// A workgroup computes a BM x BN tile of C = W X^T for one expert: W (the A
// operand) is BM output features of the expert's packed weights, X (the B
// operand) is BN of the expert's token rows (K contiguous).  Four waves split
// the features (4 x 128); each wave owns a 128-feature x 128-token block, so
// 64 MFMA blocks of 16 x 16 per 32-wide K step.
//
//  - A never touches LDS: the packed layout already holds every 16 x 32
//    fragment as 1 KiB in lane order, each fragment is used by exactly one
//    wave, and the wave loads it straight into registers two K stages ahead.
//  - B (the gathered token rows, shared by all four waves) is staged through
//    double-buffered LDS in the same fragment order, loaded two stages ahead
//    into registers, so the only LDS traffic is one 16 KiB write and four
//    16 KiB reads per 64-wide K stage.
//  - Token blocks past the expert's last row skip their MFMAs, so the padding
//    waste is at most 15 rows per expert instead of a whole tile.
//  - Workgroups are numbered so that consecutive tiles (same weight slab,
//    consecutive token tiles) land on the same XCD and share its L2.
//
// gemm<kGateUp>: A = GU slab (gate and up row tiles interleaved), X = the
//   expert's rows of x gathered through row_token; epilogue
//   H = bf16(silu(G) * U) (paper Table tab:vars (e): w1 gate, v1 up).
// gemm<kDown>:   A = DN slab, X = the expert's rows of H; epilogue O fp32.
//
// Token tiles (expert, first grouped row) come from the routing kernel; the
// grid is sized for the worst case and surplus workgroups exit at once.
#include "moe_common.h"

namespace moe {

constexpr int BM = 512;         // features per workgroup tile
constexpr int BN = 128;         // token rows per workgroup tile
constexpr int BK = 64;          // K per stage (two 32-K fragments)
constexpr int kThreads = 256;   // 4 waves, one per 128-feature slab
constexpr int FB = 8;           // 16-feature blocks per wave
constexpr int NB = BN / 16;     // 16-token blocks per tile
constexpr int B_FRAGS = NB * (BK / 32);           // 16 fragments of B per stage
constexpr int B_LOADS = B_FRAGS * 64 / kThreads;  // 4 per thread
constexpr int B_STAGE_BYTES = B_FRAGS * kTileBytes;  // 16 KiB
constexpr int kXcds = 8;

enum { kGateUp = 0, kDown = 1 };

template <int kMode>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs a)
{
    __shared__ __attribute__((aligned(16))) uint8_t lds[2][B_STAGE_BYTES];
    const int M = kMode == kGateUp ? 2 * a.f : a.d;    // a multiple of 128
    const int n_ftiles = (M + BM - 1) / BM;
    // XCD-aware numbering: hardware hands block b to XCD b % 8; give each XCD
    // a contiguous run of logical tiles.
    const int nblk = gridDim.x;
    const int per_xcd = nblk / kXcds;
    const int logical = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    const int ft = logical / a.max_tiles;
    const int tt = logical % a.max_tiles;
    if (ft >= n_ftiles || tt >= *a.n_tiles) return;
    const int e = a.tiles[2 * tt];
    const int row_start = a.tiles[2 * tt + 1];
    const int row_end = min(row_start + BN, a.offsets[e + 1]);
    const int nbv = (row_end - row_start + 15) / 16;   // token blocks with rows

    const int K = kMode == kGateUp ? a.d : a.f;
    const uint64_t KT = (uint64_t)K / kTileK;
    const int n_stages = K / BK;
    const uint8_t* wbase = a.experts + (uint64_t)(e - a.e_begin) * a.expert_bytes +
                           (kMode == kGateUp ? 0 : a.gu_bytes);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    // in a partial last feature tile, waves past M recompute the last valid
    // slab (loads stay unconditional) and skip their stores
    const bool wave_on = (uint64_t)ft * (BM / 16) + w * FB < (uint64_t)(M / 16);
    const uint64_t rt0 = wave_on ? (uint64_t)ft * (BM / 16) + w * FB : (uint64_t)(M / 16 - FB);

    // A: fragment (fb, ks) of stage s at a_src[fb] + (2s + ks) KiB
    const uint8_t* a_src[FB];
#pragma unroll
    for (int fb = 0; fb < FB; ++fb) a_src[fb] = wbase + tile_offset(rt0 + fb, 0, KT) + lane * 16;
    // B: this thread's fragments fr = w + 4 i -> (token block fr / 2, K half fr % 2)
    const uint16_t* b_src[B_LOADS];
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
        const int fr = w + 4 * i;
        const int row = row_start + (fr / 2) * 16 + (lane & 15);
        const int rr = row < row_end ? row : row_start;   // rows past the end: any valid row
        const int kofs = (fr % 2) * 32 + (lane >> 4) * 8;
        if (kMode == kGateUp)
            b_src[i] = a.x + (int64_t)a.row_token[rr] * a.d + kofs;
        else
            b_src[i] = a.H + (int64_t)rr * a.f + kofs;
    }

    f32x4_t acc[FB][NB];
#pragma unroll
    for (int fb = 0; fb < FB; ++fb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[fb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    u32x4_t ra[2][FB * 2];
    u32x4_t rb[2][B_LOADS];
    auto load = [&](int s, u32x4_t (&A)[FB * 2], u32x4_t (&B)[B_LOADS]) {
#pragma unroll
        for (int fb = 0; fb < FB; ++fb)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
                A[fb * 2 + ks] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(
                    a_src[fb] + (uint64_t)(2 * s + ks) * kTileBytes));
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i)
            B[i] = *reinterpret_cast<const u32x4_t*>(b_src[i] + s * BK);
    };
    auto store_b = [&](int buf, const u32x4_t (&B)[B_LOADS]) {
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i)
            *reinterpret_cast<u32x4_t*>(&lds[buf][(w + 4 * i) * kTileBytes + lane * 16]) = B[i];
    };
    auto compute = [&](int buf, const u32x4_t (&A)[FB * 2]) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            u32x4_t fbv[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                fbv[nb] = *reinterpret_cast<const u32x4_t*>(
                    &lds[buf][(nb * 2 + ks) * kTileBytes + lane * 16]);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                if (nb < nbv) {
#pragma unroll
                    for (int fb = 0; fb < FB; ++fb)
                        acc[fb][nb] = mfma16x16x32(A[fb * 2 + ks], fbv[nb], acc[fb][nb]);
                }
            }
        }
    };

    // prologue: stages 0 and 1 in flight, B(0) staged
    load(0, ra[0], rb[0]);
    load(1, ra[1], rb[1]);
    store_b(0, rb[0]);
    __syncthreads();
    // n_stages is even (K is a multiple of 128): iterate in pairs so that the
    // register double buffers are indexed statically
    // (the last two iterations reload the final stages: unconditional loads
    // keep the wait counts exact)
    for (int s = 0; s < n_stages; s += 2) {
        compute(0, ra[0]);
        load(min(s + 2, n_stages - 2), ra[0], rb[0]);
        store_b(1, rb[1]);
        __syncthreads();
        compute(1, ra[1]);
        load(min(s + 3, n_stages - 1), ra[1], rb[1]);
        store_b(0, rb[0]);
        __syncthreads();
    }

    // epilogue: lane holds features 4*(lane/16)+r of token column lane%16
    if (!wave_on) return;
    const int g = lane >> 4;
    const int jcol = lane & 15;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int row = row_start + nb * 16 + jcol;
        if (row >= row_end) continue;
        if (kMode == kGateUp) {
#pragma unroll
            for (int fb = 0; fb < FB; fb += 2) {
                const f32x4_t gg = acc[fb][nb], uu = acc[fb + 1][nb];
                const int feat = (int)((rt0 + fb) / 2) * 16 + g * 4;
                uint32_t h01 = (uint32_t)f32_to_bf16(silu_mul(gg[0], uu[0])) |
                               ((uint32_t)f32_to_bf16(silu_mul(gg[1], uu[1])) << 16);
                uint32_t h23 = (uint32_t)f32_to_bf16(silu_mul(gg[2], uu[2])) |
                               ((uint32_t)f32_to_bf16(silu_mul(gg[3], uu[3])) << 16);
                *reinterpret_cast<uint2*>(a.H + (int64_t)row * a.f + feat) = make_uint2(h01, h23);
            }
        } else {
#pragma unroll
            for (int fb = 0; fb < FB; ++fb) {
                const f32x4_t o = acc[fb][nb];
                const int feat = (int)(rt0 + fb) * 16 + g * 4;
                *reinterpret_cast<float4*>(a.O + (int64_t)row * a.d + feat) =
                    make_float4(o[0], o[1], o[2], o[3]);
            }
        }
    }
}

}  // namespace moe

extern "C" int moe_prefill_tile_rows() { return moe::BN; }

static int gemm_grid(int n_ftiles, int max_tiles)
{
    const int n = n_ftiles * max_tiles;
    return (n + moe::kXcds - 1) / moe::kXcds * moe::kXcds;
}

extern "C" hipError_t moe_launch_gemm_gateup(const moe::GemmArgs* a, hipStream_t s)
{
    const int grid = gemm_grid((2 * a->f + moe::BM - 1) / moe::BM, a->max_tiles);
    hipLaunchKernelGGL(moe::gemm_kernel<moe::kGateUp>, dim3(grid), dim3(moe::kThreads), 0, s, *a);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_gemm_down(const moe::GemmArgs* a, hipStream_t s)
{
    const int grid = gemm_grid((a->d + moe::BM - 1) / moe::BM, a->max_tiles);
    hipLaunchKernelGGL(moe::gemm_kernel<moe::kDown>, dim3(grid), dim3(moe::kThreads), 0, s, *a);
    return hipGetLastError();
}

extern "C" hipError_t moe_prefill_set_lds_limit() { return hipSuccess; }
