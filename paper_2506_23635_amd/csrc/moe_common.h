// moe_common.h -- shared device helpers and the packed weight layout of the
// gfx950 MoE library.
//
// Packed ("fragment-tiled") weight layout
// ---------------------------------------
// Every expert matrix is stored with its output features as rows and its
// reduction dimension K contiguous, cut into 16-row x 32-K tiles of 1 KiB.
// Inside a tile, 16-byte granule g (0..63) holds the 8 consecutive K values
// k = 8*(g/16) .. 8*(g/16)+7 of row g%16, which is exactly the bf16 operand a
// lane of a wave supplies to v_mfma_f32_16x16x32_bf16 (lane l: row l%16,
// K-group l/16).  A row tile's K tiles are consecutive, so a 16-row slab is
// one contiguous run and every wave-wide 16-byte load is 1 KiB contiguous.
//
//   GU (gate+up)  : 2*f rows x d K. Row tile 2b holds gate (w1) features
//                   16b..16b+15, row tile 2b+1 the up (v1) features of the
//                   same indices, so one wave owns both halves of a SiLU pair.
//   DN (down)     : d rows x f K, row tile q holds output features 16q..16q+15.
//
// Arena per layer: router wrT fp32 [E,d] (transposed) | bias fp32 [E] (padded) | for each
// local expert: GU then DN.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;

constexpr int kTileRows = 16;
constexpr int kTileK = 32;
constexpr int kTileBytes = kTileRows * kTileK * 2;  // 1 KiB
constexpr int kWave = 64;

// Packed row of feature n of a matrix whose rows come in heads of width hd
// (a multiple of 32) to be rotated in pairs (i, i + hd/2): tile m of a head
// holds features 8m .. 8m+7 in rows 0..7 and hd/2 + 8m .. +7 in rows 8..15,
// so both members of a pair sit in one 16-row tile, 8 rows apart.
__host__ __device__ inline int rope_row(int n, int hd)
{
    const int i = n % hd, half = hd / 2;
    const int r = i < half ? (i / 8) * 16 + i % 8 : ((i - half) / 8) * 16 + 8 + (i - half) % 8;
    return n - i + r;
}

// Byte offset of (row tile rt, K tile kt) for a matrix with KT K tiles.
__host__ __device__ inline uint64_t tile_offset(uint64_t rt, uint64_t kt, uint64_t KT)
{
    return (rt * KT + kt) * (uint64_t)kTileBytes;
}

__device__ inline float bf16_to_f32(uint16_t b)
{
    return __uint_as_float((uint32_t)b << 16);
}

// fp32 -> bf16, round to nearest even (inputs here are finite).
__device__ inline uint16_t f32_to_bf16(float v)
{
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7F800000u) == 0x7F800000u)  // inf / nan: keep, quiet the nan
        return (uint16_t)((u >> 16) | ((u & 0x007FFFFFu) ? 0x40u : 0u));
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Two fp32 -> packed bf16 (lo in the low half) by the hardware conversion:
// round to nearest even, equal to f32_to_bf16 on every non-NaN input; a NaN
// stays a NaN.
__device__ inline uint32_t cvt_pk_bf16(float lo, float hi)
{
    typedef float f32x2_v __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
    const f32x2_v in = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(in, bf16x2_v));
}

// silu(g) * u with an overflow-free logistic: for g << 0, exp(-g) -> inf,
// 1 / inf -> 0 and g * 0 -> -0, which is the limit.  The reciprocal is the
// hardware one (1 ulp): the result is rounded to bf16 next.
__device__ inline float silu_mul(float g, float u)
{
    return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

__device__ inline f32x4_t mfma16x16x32(const u32x4_t a, const u32x4_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// Workspace routing block shared by the kernels (device pointers).
struct RouteView {
    float* logits;        // [Tm, E]
    int32_t* topk_idx;    // [Tm, k]
    float* topk_w;        // [Tm, k]
    int32_t* counts;      // [E]
    int32_t* offsets;     // [E + 1]
    int32_t* pair_row;    // [Tm * k]
    int32_t* row_token;   // [Tm * k]
    int32_t* active;      // [E + 1]: active[0] = #local experts with tokens, then their ids
    int32_t* tiles;       // [max_tiles * 2]: (expert, first row) per token tile; [.. ] count
    int32_t* n_tiles;     // [1]
};

// Arguments of the decode expert kernels (moe_decode.hip).
struct DecodeArgs {
    const uint8_t* experts;   // arena: first local expert of this layer
    uint64_t expert_bytes;    // stride between local experts
    uint64_t gu_bytes;        // offset of DN inside an expert
    const uint16_t* x;        // [T, d]
    uint16_t* H;              // [rows, f]
    float* O;                 // [rows, d]
    const int32_t* active;    // [1 + E]
    const int32_t* counts;    // [E]
    const int32_t* offsets;   // [E + 1]
    const int32_t* row_token; // [rows]
    int d, f, e_begin;
};

// Arguments of the prefill grouped GEMM kernels (moe_prefill.hip).
struct GemmArgs {
    const uint8_t* experts;   // arena: first local expert of this layer
    uint64_t expert_bytes;
    uint64_t gu_bytes;
    const uint16_t* x;        // [T, d]
    uint16_t* H;              // [rows, f]
    float* O;                 // [rows, d]
    const int32_t* offsets;   // [E + 1]
    const int32_t* row_token; // [rows]
    const int32_t* tiles;     // [max_tiles][2] = (expert, first row)
    const int32_t* n_tiles;   // [1]
    int d, f, e_begin, max_tiles;
    int T;                    // tokens of the call (rows of x)
    uint64_t* stamps;         // per-workgroup timeline [max_stamps][8], or NULL (measurement)
    int max_stamps;
};

}  // namespace moe

// Launchers (one per kernel family); each returns the launch status.
extern "C" {
hipError_t moe_launch_pack(const uint16_t* src, int K, int N, void* dst, int rt_mul, int rt_add,
                           hipStream_t s);
void moe_pack_host(const uint16_t* src, int K, int N, uint8_t* dst, int rt_mul, int rt_add);
hipError_t moe_launch_pack_perm(const uint16_t* src, int K, int N, void* dst, int rt_mul,
                                int rt_add, int perm_hd, int perm_rows, hipStream_t s);
void moe_pack_host_perm(const uint16_t* src, int K, int N, uint8_t* dst, int rt_mul, int rt_add,
                        int perm_hd, int perm_rows);
int moe_route_decode_ok(int T, int E, int k);
int moe_route_decode_wgs(int d);
hipError_t moe_launch_route_decode(const uint16_t* x, const float* wrT, const float* bias,
                                   double* partial, int T, int d, int E, int k, int e_begin,
                                   int n_local, int tile_rows,
                                   const moe::RouteView* rv, hipStream_t s);
hipError_t moe_launch_router_select(const uint16_t* x, const float* wrT, const float* bias, int T,
                                   int d, int E, int k, const moe::RouteView* rv, hipStream_t s);
hipError_t moe_launch_route(const float* logits_in, int T, int E, int k, int e_begin, int n_local,
                            int tile_rows, const moe::RouteView* rv, hipStream_t s);
hipError_t moe_launch_transpose_router(const float* wr, int d, int E, float* wrT, hipStream_t s);
hipError_t moe_launch_decode_gateup(const moe::DecodeArgs* a, int n_slots, hipStream_t s);
hipError_t moe_launch_decode_down(const moe::DecodeArgs* a, int n_slots, hipStream_t s);
hipError_t moe_launch_gemm_gateup(const moe::GemmArgs* a, hipStream_t s);
hipError_t moe_launch_gemm_down(const moe::GemmArgs* a, hipStream_t s);
int moe_prefill_tile_rows();
hipError_t moe_launch_combine(const float* O, const int32_t* pair_row, const float* topk_w, int T,
                              int d, int k, uint16_t* y, float* y32, uint16_t* x_residual,
                              hipStream_t s);
}

// Launchers of the attention-block kernels (attn.hip).
extern "C" {
hipError_t attn_launch_norm(const uint16_t* x, const float* gamma, int T, int d, float eps,
                            uint16_t* h, hipStream_t s);
int attn_norm_in_projection(int T);
hipError_t attn_launch_qkv(const void* w, uint16_t* h, const uint16_t* x, const float* gamma,
                           float eps, const double* inv_freq, float* qkv, uint16_t* q,
                           uint16_t* kc, uint16_t* vc, int T, int d, int H, int G, int hd,
                           int max_seq, int pos0, hipStream_t s);
hipError_t attn_launch_out(const void* w, const uint16_t* x, int T, int K, int N, float* y32,
                           const uint16_t* res, uint16_t* y16, hipStream_t s);
hipError_t attn_launch_rope(const float* qkvp, const double* inv_freq, float* qkv, uint16_t* q,
                            uint16_t* kc, uint16_t* vc, int T, int H, int G, int hd, int max_seq,
                            int pos0, hipStream_t s);
hipError_t attn_launch_flash(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                             uint16_t* out, int T, int H, int G, int hd, int max_seq, int pos0,
                             hipStream_t s);
hipError_t attn_launch_residual(const uint16_t* x, const float* o, uint16_t* y, int64_t n,
                                hipStream_t s);
int attn_chunks(int n_pos);
int attn_part_stride(int hd);
hipError_t attn_launch_score(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                             float* part, int T, int H, int G, int hd, int max_seq, int pos0,
                             int n_chunks_alloc, hipStream_t s);
hipError_t attn_launch_combine(const float* part, uint16_t* out, int T, int H, int hd, int pos0,
                               int n_chunks_alloc, hipStream_t s);
}
