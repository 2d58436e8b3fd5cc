// moe_prefill.hip -- the expert FFN for many tokens (prefill): a grouped GEMM
// on the bf16 matrix cores (v_mfma_f32_16x16x32_bf16).
//
// One workgroup computes a BM x BN tile of C = W * X^T for one expert, where
// the A operand W is a slab of the expert's packed weights (BM output features
// x K, already in MFMA fragment order in HBM) and the B operand X holds BN of
// the expert's token rows (K contiguous).  Both operands are staged through
// LDS in 16 x 32 fragments of 1 KiB (lane l owns row l%16, K group l/16), so
// every LDS read and write is a conflict-free contiguous 16 bytes per lane.
// The K loop is double-buffered: the global loads of stage s+1 are in flight
// while stage s feeds the matrix cores.
//
// gemm<kGateUp>: A = GU slab (gate and up row tiles interleaved), X = the
//   expert's token rows of x gathered through row_token; epilogue
//   H = bf16(silu(G) * U) (paper Table tab:vars (e): w1 gate, v1 up).
// gemm<kDown>:   A = DN slab, X = the expert's rows of H; epilogue O fp32.
//
// Token tiles (expert, first grouped row) come from the routing kernel; the
// grid is sized for the worst case and surplus workgroups exit at once.
#include "moe_common.h"

namespace moe {

constexpr int BM = 256;         // features per tile
constexpr int BN = 128;         // token rows per tile
constexpr int BK = 64;          // K per stage (two 32-K fragments)
constexpr int kThreads = 256;   // 4 waves: 2 (features) x 2 (tokens)
constexpr int WM = BM / 2;      // 128 features per wave
constexpr int WN = BN / 2;      // 64 tokens per wave
constexpr int MB = WM / 16;     // 8 MFMA row blocks per wave
constexpr int NB = WN / 16;     // 4 MFMA column blocks per wave
constexpr int A_FRAGS = (BM / 16) * (BK / 32);   // 32
constexpr int B_FRAGS = (BN / 16) * (BK / 32);   // 16
constexpr int A_LOADS = A_FRAGS * 64 / kThreads;  // 8 per thread
constexpr int B_LOADS = B_FRAGS * 64 / kThreads;  // 4 per thread
constexpr int STAGE_BYTES = (A_FRAGS + B_FRAGS) * kTileBytes;  // 48 KiB

enum { kGateUp = 0, kDown = 1 };

template <int kMode>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs a)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    const int n_ftiles = (kMode == kGateUp ? 2 * a.f : a.d) / BM;
    const int ft = blockIdx.x / a.max_tiles;
    const int tt = blockIdx.x % a.max_tiles;
    if (ft >= n_ftiles || tt >= *a.n_tiles) return;
    const int e = a.tiles[2 * tt];
    const int row_start = a.tiles[2 * tt + 1];
    const int row_end = min(row_start + BN, a.offsets[e + 1]);

    const int K = kMode == kGateUp ? a.d : a.f;
    const uint64_t KT = (uint64_t)K / kTileK;
    const int n_stages = K / BK;
    const uint8_t* wbase = a.experts + (uint64_t)(e - a.e_begin) * a.expert_bytes +
                           (kMode == kGateUp ? 0 : a.gu_bytes);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wm = wid >> 1;
    const int wn = wid & 1;

    // A chunks: fragment fr = tid/64 + 4*i -> (row tile fr/2, K half fr%2)
    const uint8_t* a_src[A_LOADS];
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
        const int fr = (tid >> 6) + 4 * i;
        a_src[i] = wbase + tile_offset((uint64_t)ft * (BM / 16) + fr / 2, fr % 2, KT) + lane * 16;
    }
    // B chunks: fragment fr = tid/64 + 4*i -> (token row tile fr/2, K half fr%2)
    const uint16_t* b_src[B_LOADS];
    bool b_ok[B_LOADS];
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
        const int fr = (tid >> 6) + 4 * i;
        const int row = row_start + (fr / 2) * 16 + (lane & 15);
        const int kofs = (fr % 2) * 32 + (lane >> 4) * 8;
        b_ok[i] = row < row_end;
        const int rr = b_ok[i] ? row : row_start;
        if (kMode == kGateUp)
            b_src[i] = a.x + (int64_t)a.row_token[rr] * a.d + kofs;
        else
            b_src[i] = a.H + (int64_t)rr * a.f + kofs;
    }

    u32x4_t ra[A_LOADS], rb[B_LOADS];
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    auto load_stage = [&](int s) {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i)
            ra[i] = __builtin_nontemporal_load(
                reinterpret_cast<const u32x4_t*>(a_src[i] + (uint64_t)s * 2 * kTileBytes));
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i)
            rb[i] = b_ok[i] ? *reinterpret_cast<const u32x4_t*>(b_src[i] + s * BK) : zero;
    };
    auto store_stage = [&](int buf) {
        uint8_t* base = lds + buf * STAGE_BYTES;
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i)
            *reinterpret_cast<u32x4_t*>(base + ((tid >> 6) + 4 * i) * kTileBytes + lane * 16) = ra[i];
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i)
            *reinterpret_cast<u32x4_t*>(base + (A_FRAGS + (tid >> 6) + 4 * i) * kTileBytes +
                                        lane * 16) = rb[i];
    };

    f32x4_t acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int s = 0; s < n_stages; ++s) {
        const int buf = s & 1;
        if (s + 1 < n_stages) load_stage(s + 1);
        const uint8_t* base = lds + buf * STAGE_BYTES;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            u32x4_t fa[MB], fb[NB];
#pragma unroll
            for (int i = 0; i < MB; ++i)
                fa[i] = *reinterpret_cast<const u32x4_t*>(
                    base + ((wm * MB + i) * 2 + ks) * kTileBytes + lane * 16);
#pragma unroll
            for (int j = 0; j < NB; ++j)
                fb[j] = *reinterpret_cast<const u32x4_t*>(
                    base + (A_FRAGS + (wn * NB + j) * 2 + ks) * kTileBytes + lane * 16);
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int j = 0; j < NB; ++j) acc[i][j] = mfma16x16x32(fa[i], fb[j], acc[i][j]);
        }
        if (s + 1 < n_stages) store_stage(buf ^ 1);
        __syncthreads();
    }

    // epilogue: lane holds features 4*(lane/16)+r of token column lane%16
    const int g = lane >> 4;
    const int jcol = lane & 15;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int row = row_start + wn * WN + j * 16 + jcol;
        if (row >= row_end) continue;
        if (kMode == kGateUp) {
#pragma unroll
            for (int i = 0; i < MB; i += 2) {
                const f32x4_t gg = acc[i][j], uu = acc[i + 1][j];
                const int feat = (ft * (BM / 32) + wm * (MB / 2) + i / 2) * 16 + g * 4;
                uint32_t h01 = (uint32_t)f32_to_bf16(silu_mul(gg[0], uu[0])) |
                               ((uint32_t)f32_to_bf16(silu_mul(gg[1], uu[1])) << 16);
                uint32_t h23 = (uint32_t)f32_to_bf16(silu_mul(gg[2], uu[2])) |
                               ((uint32_t)f32_to_bf16(silu_mul(gg[3], uu[3])) << 16);
                *reinterpret_cast<uint2*>(a.H + (int64_t)row * a.f + feat) = make_uint2(h01, h23);
            }
        } else {
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                const f32x4_t o = acc[i][j];
                const int feat = (ft * (BM / 16) + wm * MB + i) * 16 + g * 4;
                *reinterpret_cast<float4*>(a.O + (int64_t)row * a.d + feat) =
                    make_float4(o[0], o[1], o[2], o[3]);
            }
        }
    }
}

}  // namespace moe

extern "C" int moe_prefill_tile_rows() { return moe::BN; }

extern "C" hipError_t moe_launch_prefill(const moe::GemmArgs* a, hipStream_t s)
{
    const size_t lds_bytes = 2 * moe::STAGE_BYTES;
    const int gu_blocks = (2 * a->f / moe::BM) * a->max_tiles;
    const int dn_blocks = (a->d / moe::BM) * a->max_tiles;
    hipLaunchKernelGGL(moe::gemm_kernel<moe::kGateUp>, dim3(gu_blocks), dim3(moe::kThreads),
                       lds_bytes, s, *a);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(moe::gemm_kernel<moe::kDown>, dim3(dn_blocks), dim3(moe::kThreads),
                       lds_bytes, s, *a);
    return hipGetLastError();
}

extern "C" hipError_t moe_prefill_set_lds_limit()
{
    const int lds_bytes = 2 * moe::STAGE_BYTES;
    hipError_t e1 = hipFuncSetAttribute((const void*)moe::gemm_kernel<moe::kGateUp>,
                                        hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    hipError_t e2 = hipFuncSetAttribute((const void*)moe::gemm_kernel<moe::kDown>,
                                        hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    return e1 != hipSuccess ? e1 : e2;
}
