// moe_prefill.hip -- the expert FFN for many tokens (prefill): a grouped GEMM
// on the bf16 matrix cores (v_mfma_f32_16x16x32_bf16).
//
// A workgroup computes a BM x BN tile of C = W X^T for one expert: W (the A
// operand) is BM output features of the expert's packed weights, X (the B
// operand) is BN of the expert's token rows (K contiguous).  Four waves split
// the features (4 x 64); each wave owns a 64-feature x 256-token block, so 64
// MFMA blocks of 16 x 16 per 32-wide K step, and each weight slab is re-read
// by only ceil(tokens / 256) workgroups.
//
//  - A never touches LDS: the packed layout already holds every 16 x 32
//    fragment as 1 KiB in lane order, each fragment is used by exactly one
//    wave, and the wave loads it straight into registers through a ring of
//    three K stages (two in flight while one computes).
//  - B (the gathered token rows, shared by all four waves) is staged through
//    double-buffered LDS in the same fragment order, loaded two stages ahead
//    into registers, so the only LDS traffic is one 32 KiB write and four
//    32 KiB reads per 64-wide K stage.
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

constexpr int BM = 256;         // features per workgroup tile
constexpr int BN = 256;         // token rows per workgroup tile
constexpr int BK = 64;          // K per stage (two 32-K fragments)
constexpr int kThreads = 256;   // 4 waves, one per 64-feature slab
constexpr int FB = 4;           // 16-feature blocks per wave
constexpr int NB = BN / 16;     // 16-token blocks per tile
constexpr int A_STAGES = 3;     // register ring of A stages (two in flight while one computes)
constexpr int B_FRAGS = NB * (BK / 32);           // 32 fragments of B per stage
constexpr int B_LOADS = B_FRAGS * 64 / kThreads;  // 8 per thread
constexpr int B_STAGE_BYTES = B_FRAGS * kTileBytes;  // 32 KiB
constexpr int B_BUFS = 3;       // LDS ring of B stages (two in flight while one computes)
constexpr int kXcds = 8;
constexpr int kBBatch = 4;      // B fragments read from LDS per MFMA batch
// s_waitcnt immediate (gfx9 layout: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] |
// vmcnt[15:14]) waiting until at most N vector-memory ops are outstanding:
// before stage s the ops issued after B(s) are B(s+1) and A(s+1), A(s+2).
constexpr int kAfterB = B_LOADS + 2 * (FB * 2);   // 8 + 16 = 24
constexpr int kWaitAll = (0x7 << 4) | (0xF << 8);   // vmcnt 0
constexpr int kWaitBStage = (kAfterB & 0xF) | ((kAfterB >> 4) << 14) | (0x7 << 4) | (0xF << 8);

enum { kGateUp = 0, kDown = 1 };

struct TileCtx {
    const uint8_t* a_src;      // this lane's first A fragment (stage 0, ks 0)
    uint64_t a_fstride;        // bytes between 16-feature blocks
    const uint16_t* b_base;    // x (gathered) or H
    uint32_t b_off[B_LOADS];   // element offsets of this thread's B rows
    int n_stages;
    int w, lane;
};

// The K loop of one tile.  Token blocks go in batches of kBBatch; only the
// first n_batch batches (those holding rows of the tile) run their MFMAs, and
// the check is one uniform branch per batch of 16 MFMAs.
__device__ __forceinline__ void tile_loop(const TileCtx& c, int n_batch, uint8_t* lds,
                                          f32x4_t (&acc)[FB][NB])
{
    constexpr int kNb = NB;
    const int n_stages = c.n_stages;
    const int w = c.w, lane = c.lane;
    u32x4_t ra[A_STAGES][FB * 2];
    auto load_a = [&](int s, u32x4_t (&A)[FB * 2]) {
#pragma unroll
        for (int fb = 0; fb < FB; ++fb)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
                A[fb * 2 + ks] = *reinterpret_cast<const u32x4_t*>(
                    c.a_src + fb * c.a_fstride + (uint64_t)(2 * s + ks) * kTileBytes);
    };
    // B goes global -> LDS directly (16 bytes per lane; a wave-wide load
    // fills one 1 KiB fragment in lane order)
    auto load_b = [&](int s, int buf) {
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i)
            __builtin_amdgcn_global_load_lds(
                (__attribute__((address_space(1))) const void*)(c.b_base + c.b_off[i] + s * BK),
                (__attribute__((address_space(3))) void*)(&lds[buf * B_STAGE_BYTES +
                                                               (w + 4 * i) * kTileBytes]),
                16, 0, 0);
    };
    // B fragments are read from LDS in batches of kBBatch, one batch ahead of
    // the MFMAs that use it (sched_barrier keeps the scheduler from hoisting
    // more reads than that and running out of registers)
    constexpr int kBatches = 2 * (kNb / kBBatch);   // (K half, token batch) pairs
    auto batch_on = [&](int bi) { return (bi % (kNb / kBBatch)) < n_batch; };
    auto read_batch = [&](int buf, int bi, u32x4_t (&B)[kBBatch]) {
        const int ks = bi / (kNb / kBBatch);
        const int nh = (bi % (kNb / kBBatch)) * kBBatch;
#pragma unroll
        for (int q = 0; q < kBBatch; ++q)
            B[q] = *reinterpret_cast<const u32x4_t*>(
                &lds[buf * B_STAGE_BYTES + ((nh + q) * 2 + ks) * kTileBytes + lane * 16]);
    };
    auto compute = [&](int buf, const u32x4_t (&A)[FB * 2]) {
        u32x4_t bb[2][kBBatch];
        read_batch(buf, 0, bb[0]);
#pragma unroll
        for (int bi = 0; bi < kBatches; ++bi) {
            if (bi + 1 < kBatches) read_batch(buf, bi + 1, bb[(bi + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            const int ks = bi / (kNb / kBBatch);
            const int nh = (bi % (kNb / kBBatch)) * kBBatch;
            if (batch_on(bi)) {
#pragma unroll
                for (int q = 0; q < kBBatch; ++q)
#pragma unroll
                    for (int fb = 0; fb < FB; ++fb)
                        acc[fb][nh + q] =
                            mfma16x16x32(A[fb * 2 + ks], bb[bi & 1][q], acc[fb][nh + q]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // prologue: A stages 0..2 in registers, B stages 0..1 in LDS, in flight
    load_b(0, 0);
    load_a(0, ra[0]);
    load_b(1, 1);
    load_a(1, ra[1]);
    load_a(2, ra[2]);
    // One iteration = three stages, so that both rings are indexed
    // statically.  Before stage s: wait for this wave's B(s) (everything but
    // the B(s+1), A(s+1), A(s+2) issued after it) and barrier, so every
    // wave's B(s) is in LDS and every wave is done reading B(s-1)'s buffer;
    // then issue B(s+2) into that buffer, compute stage s, refill ra[s % 3]
    // with A(s+3).  Loads past the last stage re-read the last stage.
    auto step = [&](int s, u32x4_t (&A)[FB * 2], int buf) {
        // explicit partial wait + bare barrier: a __syncthreads() release
        // fence would wait for every outstanding LDS DMA (vmcnt 0); the empty
        // asm statements keep the compiler from moving memory operations
        // across the barrier
        __builtin_amdgcn_s_waitcnt(kWaitBStage);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        load_b(min(s + 2, n_stages - 1), (buf + 2) % 3);
        compute(buf, A);
        load_a(min(s + 3, n_stages - 1), A);
    };
    int s = 0;
    for (; s + 3 <= n_stages; s += 3) {
        step(s + 0, ra[0], 0);
        step(s + 1, ra[1], 1);
        step(s + 2, ra[2], 2);
    }
    if (s < n_stages) step(s++, ra[0], 0);
    if (s < n_stages) step(s++, ra[1], 1);
    // the last steps re-issued dummy B loads into LDS: drain them before the
    // workgroup can finish and its LDS be handed to another workgroup
    __builtin_amdgcn_s_waitcnt(kWaitAll);
    __builtin_amdgcn_s_barrier();
}

template <int kMode>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs a)
{
    __shared__ __attribute__((aligned(16))) uint8_t lds[B_BUFS * B_STAGE_BYTES];
    const int M = kMode == kGateUp ? 2 * a.f : a.d;    // a multiple of 128
    const int n_ftiles = (M + BM - 1) / BM;
    // XCD-aware numbering: hardware hands block b to XCD b % 8; give each XCD
    // a contiguous run of logical tiles (token tile fastest, so the tiles
    // that share a weight slab run together on one XCD).
    const int per_xcd = gridDim.x / kXcds;
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
    const uint8_t* wbase = a.experts + (uint64_t)(e - a.e_begin) * a.expert_bytes +
                           (kMode == kGateUp ? 0 : a.gu_bytes);

    TileCtx c;
    c.n_stages = K / BK;
    c.lane = threadIdx.x & 63;
    c.w = threadIdx.x >> 6;
    const int lane = c.lane, w = c.w;
    // a wave past M (partial last feature tile) recomputes the last valid
    // slab, keeping every load unconditional, and skips its stores
    const bool wave_on = (uint64_t)ft * (BM / 16) + w * FB < (uint64_t)(M / 16);
    const uint64_t rt0 = wave_on ? (uint64_t)ft * (BM / 16) + w * FB : (uint64_t)(M / 16 - FB);
    // A: fragment (fb, ks) of stage s at a_src + fb * a_fstride + (2s + ks) KiB
    c.a_src = wbase + tile_offset(rt0, 0, KT) + lane * 16;
    c.a_fstride = KT * kTileBytes;
    // B: this thread's fragments fr = w + 4 i -> (token block fr / 2, K half
    // fr % 2), held as 32-bit element offsets into x (gathered) or H
    c.b_base = kMode == kGateUp ? a.x : a.H;
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
        const int fr = w + 4 * i;
        const int row = row_start + (fr / 2) * 16 + (lane & 15);
        const int rr = row < row_end ? row : row_start;   // rows past the end: any valid row
        const int kofs = (fr % 2) * 32 + (lane >> 4) * 8;
        if (kMode == kGateUp)
            c.b_off[i] = (uint32_t)a.row_token[rr] * (uint32_t)a.d + kofs;
        else
            c.b_off[i] = (uint32_t)rr * (uint32_t)a.f + kofs;
    }

    f32x4_t acc[FB][NB];
#pragma unroll
    for (int fb = 0; fb < FB; ++fb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[fb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    tile_loop(c, (nbv + kBBatch - 1) / kBBatch, lds, acc);

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
