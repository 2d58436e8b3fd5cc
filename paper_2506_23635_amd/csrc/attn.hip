// attn.hip -- kernels of the self-attention block of include/attn.h for a few
// new tokens (T <= 16: decode), in launch order:
//
//   norm_kernel     layer norm for more than 4 tokens, one workgroup per
//                   token (one pass, fp64 sums, fixed reduction order),
//                   h = bf16((x - mean) rstd gamma); up to 4 tokens the
//                   projection forms h itself
//   qkv_kernel      q|k|v = h Wqkv, and in its epilogue the rotary encoding
//                   of the query and key heads (angles reduced in fp64,
//                   rotation in fp32): bf16 q to the workspace, bf16 k and v
//                   appended to the cache
//   score_kernel    attention of every query head of one key/value head over
//                   one chunk of 64 positions (4 waves): scores on the matrix
//                   cores, the chunk's softmax maximum and sum, and the
//                   unnormalised weighted sum of v
//   combine_kernel  merges the chunks of each (token, head) into bf16 a
//   gemv_kernel     o = a Wo (fp32) and y = bf16(x + o)
//
// Above 16 new tokens (prefill) the block is: norm_kernel -> q|k|v on the
// grouped GEMM of moe_prefill.hip -> rope_kernel (rotation, cache append)
// -> flash_kernel (causal attention on the matrix cores) -> o = a Wo on the
// grouped GEMM -> residual_kernel.
//
// The GEMVs stream the fragment-tiled weights (the layout of moe_common.h)
// through v_mfma_f32_16x16x32_bf16 with the tokens as the B operand, as the
// MoE decode GEMVs do: one workgroup per 16 output features, its 8 waves
// splitting K (wave w takes K tiles w, w + 8, ...), wave 0 adding the
// partial fragments in wave order.  In the attention, q . k of 16 positions
// and 16 query rows is one MFMA per 32 dims; the weighted sum of v is VALU
// work, small beside the projections' weight stream.
#include "moe_common.h"

namespace attn {

using moe::f32x4_t;
using moe::u32x4_t;
using moe::kTileK;
using moe::kTileBytes;
using moe::kTileRows;

constexpr int kSplit = 8;          // waves per GEMV workgroup (K split)
constexpr int kUnroll = 8;         // K tiles per wave in flight
constexpr int kChunk = 64;         // positions per attention workgroup
constexpr int kPartPad = 4;        // m, l and padding after the hd sums of a partial

__device__ inline u32x4_t ld16_nt(const void* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}

__device__ inline u32x4_t ld16(const void* p) { return *reinterpret_cast<const u32x4_t*>(p); }

// The output projection, o = a Wo (fp32) and y = bf16(x + o), one
// workgroup per 16 output features.
struct GemvArgs {
    const uint8_t* w;      // packed weights: N/16 row tiles of K/32 tiles
    const uint16_t* x;     // [T][K] bf16
    float* y32;            // [T][N] fp32
    const uint16_t* res;   // residual [T][N] bf16
    uint16_t* y16;         // bf16(res + y) [T][N]
    int K, N, T;
};

__global__ __launch_bounds__(64 * kSplit) void gemv_kernel(GemvArgs a)
{
    __shared__ f32x4_t s_red[(kSplit - 1) * 64];
    const int q = blockIdx.x;                   // output features 16q .. 16q+15
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int j = lane & 15, g = lane >> 4;    // token column, K group of 8
    const int KT = a.K / kTileK;
    const uint8_t* pw = a.w + moe::tile_offset(q, 0, KT) + lane * 16;
    const bool has_tok = j < a.T;
    const uint16_t* px = a.x + (has_tok ? (int64_t)j * a.K : 0) + g * 8;
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    constexpr int kStep = kSplit * kUnroll;
    const int nb = KT / kStep;                 // full batches of kUnroll tiles per wave
    // token loads without branches (an unused column reads token 0's row and
    // feeds zeros), so that a wait for them is not a wait for everything
    auto xload = [&](int k0, u32x4_t* xv) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const u32x4_t v = ld16(px + (k0 + w + kSplit * u) * kTileK);
            xv[u] = has_tok ? v : zero;
        }
    };
    auto wload = [&](int k0, u32x4_t* wt) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            wt[u] = ld16_nt(pw + (int64_t)(k0 + w + kSplit * u) * kTileBytes);
    };
    auto mfmas = [&](const u32x4_t* wt, const u32x4_t* xv) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc = moe::mfma16x16x32(wt[u], xv[u], acc);
    };
    int kt = 0;
    if (nb > 0) {
        // two weight buffers in turn: the next batch's weights are issued
        // after this batch's token loads and before its MFMAs, so they stay
        // in flight while it is multiplied
        u32x4_t wa[kUnroll], wb[kUnroll], xv[kUnroll];
        wload(0, wa);
        int b = 0;
        for (; b + 2 < nb; b += 2) {
            xload(b * kStep, xv);
            wload((b + 1) * kStep, wb);
            mfmas(wa, xv);
            xload((b + 1) * kStep, xv);
            wload((b + 2) * kStep, wa);
            mfmas(wb, xv);
        }
        xload(b * kStep, xv);
        if (b + 1 < nb) {
            wload((b + 1) * kStep, wb);
            mfmas(wa, xv);
            xload((b + 1) * kStep, xv);
            mfmas(wb, xv);
        } else {
            mfmas(wa, xv);
        }
        kt = nb * kStep;
    }
    for (kt += w; kt < KT; kt += kSplit) {
        const u32x4_t wt = ld16_nt(pw + (int64_t)kt * kTileBytes);
        const u32x4_t xt = has_tok ? ld16(px + kt * kTileK) : zero;
        acc = moe::mfma16x16x32(wt, xt, acc);
    }
    if (w > 0) s_red[(w - 1) * 64 + lane] = acc;
    __syncthreads();
    if (w != 0) return;
    for (int i = 0; i + 1 < kSplit; ++i) acc += s_red[i * 64 + lane];
    if (!has_tok) return;
    // lane holds output features 16q + 4g .. +3 of token j
    const int64_t o = (int64_t)j * a.N + q * kTileRows + g * 4;
    *reinterpret_cast<float4*>(a.y32 + o) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    const uint2 r = *reinterpret_cast<const uint2*>(a.res + o);
    const float r0 = __uint_as_float(r.x << 16), r1 = __uint_as_float(r.x & 0xFFFF0000u);
    const float r2 = __uint_as_float(r.y << 16), r3 = __uint_as_float(r.y & 0xFFFF0000u);
    const uint32_t lo = (uint32_t)moe::f32_to_bf16(r0 + acc[0]) |
                        ((uint32_t)moe::f32_to_bf16(r1 + acc[1]) << 16);
    const uint32_t hi = (uint32_t)moe::f32_to_bf16(r2 + acc[2]) |
                        ((uint32_t)moe::f32_to_bf16(r3 + acc[3]) << 16);
    *reinterpret_cast<uint2*>(a.y16 + o) = make_uint2(lo, hi);
}

// Layer norm, one workgroup of 256 threads per token: the thread's 8-element
// groups of x are loaded once into registers, x and x^2 summed in fp64 (so
// E[x^2] - mean^2 loses nothing), a butterfly per wave and the 4 wave sums in
// wave order, then h = bf16((x - mean) rstd gamma) from the registers.
constexpr int kNormThreads = 256;
constexpr int kNormGroups = 4;     // 8-element groups per thread (d <= 8192)

__global__ __launch_bounds__(kNormThreads) void norm_kernel(const uint16_t* __restrict__ x,
                                                            const float* __restrict__ gamma,
                                                            int d, float eps,
                                                            uint16_t* __restrict__ h)
{
    __shared__ double red[2][kNormThreads / 64];
    const int t = blockIdx.x;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint16_t* xr = x + (int64_t)t * d;
    u32x4_t v[kNormGroups];
    double sx = 0.0, sq = 0.0;
#pragma unroll
    for (int k = 0; k < kNormGroups; ++k) {
        const int e = threadIdx.x + k * kNormThreads;
        const u32x4_t zero = {0u, 0u, 0u, 0u};
        v[k] = e < d / 8 ? ld16(xr + e * 8) : zero;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const double lo = __uint_as_float(v[k][i] << 16);
            const double hi = __uint_as_float(v[k][i] & 0xFFFF0000u);
            sx += lo + hi;
            sq = fma(lo, lo, fma(hi, hi, sq));
        }
    }
    for (int off = 32; off >= 1; off >>= 1) {
        sx += __shfl_xor(sx, off, 64);
        sq += __shfl_xor(sq, off, 64);
    }
    if (lane == 0) { red[0][w] = sx; red[1][w] = sq; }
    __syncthreads();
    const double m1 = ((red[0][0] + red[0][1]) + red[0][2]) + red[0][3];
    const double m2 = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
    const double mean = m1 / d;
    const float rstd = (float)(1.0 / sqrt(fmax(m2 / d - mean * mean, 0.0) + (double)eps));
    const float mu = (float)mean;
#pragma unroll
    for (int k = 0; k < kNormGroups; ++k) {
        const int e = threadIdx.x + k * kNormThreads;
        if (e >= d / 8) break;
        const float4 g0 = *reinterpret_cast<const float4*>(gamma + e * 8);
        const float4 g1 = *reinterpret_cast<const float4*>(gamma + e * 8 + 4);
        const float gm[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        u32x4_t out;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float lo = (__uint_as_float(v[k][i] << 16) - mu) * rstd * gm[2 * i];
            const float hi = (__uint_as_float(v[k][i] & 0xFFFF0000u) - mu) * rstd * gm[2 * i + 1];
            out[i] = (uint32_t)moe::f32_to_bf16(lo) | ((uint32_t)moe::f32_to_bf16(hi) << 16);
        }
        *reinterpret_cast<u32x4_t*>(h + (int64_t)t * d + e * 8) = out;
    }
}

// The fused projection q|k|v = h Wqkv, one workgroup per 16 packed rows (8
// waves splitting K, as gemv_kernel).  The query and key heads are packed
// with rope_row, so in the epilogue lane (token j, group g), which holds
// rows 4g..4g+3 of the tile, and lane l ^ 32 hold the two members of four
// rotation pairs: the rotation (angle formed and reduced in fp64 from the
// layer's frequency table, sincosf, product in fp32) and the bf16 rounding
// happen there, q goes to the workspace and k, v to the cache at position
// pos0 + j; the unrotated fp32 values are kept for inspection.
struct QkvArgs {
    const uint8_t* w;      // packed Wqkv, query and key heads permuted by rope_row
    const uint16_t* h;     // [T][d] bf16, the normalised input (written here when the
                           // kernel normalises x itself)
    const uint16_t* x;     // [T][d] bf16 block input (normalising kernel only)
    const float* gamma;    // [d]
    float eps;
    const double* inv_freq;  // [hd/2]: theta^(-2f/hd)
    float* qkv;            // [T][nqkv] fp32, natural order, before rotation
    uint16_t* q;           // [T][H][hd]
    uint16_t* kc;          // this layer's K cache [G][max_seq][hd]
    uint16_t* vc;          // this layer's V cache
    int d, T, H, G, hd, max_seq, pos0;
};

// cos and sin of pos * inv_freq: the angle is formed and reduced modulo 2 pi
// in fp64 (2 pi split in two parts, Cody and Waite), so sincosf only sees an
// argument within [-pi, pi]
__device__ inline void rope_cs(int pos, double inv_freq, float& c, float& s)
{
    constexpr double kTwoPiHi = 6.28318530717958623200e+00;   // 2 pi rounded to fp64
    constexpr double kTwoPiLo = 2.44929359829470635445e-16;   // 2 pi - kTwoPiHi
    constexpr double kInvTwoPi = 1.59154943091895335769e-01;
    const double ang = (double)pos * inv_freq;
    const double k = rint(ang * kInvTwoPi);
    const double r = fma(-k, kTwoPiLo, fma(-k, kTwoPiHi, ang));
    sincosf((float)r, &s, &c);
}

// barrier for LDS traffic only: waits for this wave's LDS operations, not
// for its outstanding global loads (the weight batch in flight)
__device__ __forceinline__ void lds_barrier()
{
    constexpr int kWaitLgkm = 0xC07F;   // lgkmcnt 0; vmcnt and expcnt at their maxima
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(kWaitLgkm);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

constexpr int kLnMaxT = 4;     // tokens up to which the projection normalises x itself
constexpr int kLnGroups = 2;   // 8-element groups per thread and token (d <= 8192)
constexpr int kHPad = 8;       // bf16 padding of a token row of h in LDS

// kNorm (T <= kLnMaxT): every workgroup forms the layer norm of the T tokens
// itself, into LDS, while its first weight batch is in flight -- x and gamma
// loaded first (thread i: 8-element groups i and i + 512), then the weights,
// then x and x^2 summed in fp64 (butterfly per wave, the 8 waves in order),
// h = bf16((x - mean) rstd gamma) to LDS (workgroup 0 also writes it out);
// the main loop then reads its B fragments from LDS.  Otherwise h comes from
// norm_kernel through global memory.
template <bool kNorm>
__global__ __launch_bounds__(64 * kSplit) void qkv_kernel(QkvArgs a)
{
    __shared__ f32x4_t s_red[(kSplit - 1) * 64];
    extern __shared__ __attribute__((aligned(16))) uint16_t hs[];   // kNorm: [T][d + kHPad]
    const int q = blockIdx.x;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int j = lane & 15, g = lane >> 4;
    const int KT = a.d / kTileK;
    const int hstride = a.d + kHPad;
    const uint8_t* pw = a.w + moe::tile_offset(q, 0, KT) + lane * 16;
    const bool has_tok = j < a.T;
    const uint16_t* px = a.h + (has_tok ? (int64_t)j * a.d : 0) + g * 8;
    const uint16_t* hx = hs + (has_tok ? j * hstride : 0) + g * 8;
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    u32x4_t wv[kUnroll], xb[kUnroll];
    if constexpr (kNorm) {
        __shared__ double red[2][kLnMaxT][kSplit];
        const int tid = threadIdx.x, ng = a.d / 8;
        u32x4_t xv[kLnMaxT][kLnGroups];
        float4 gv[kLnGroups][2];
        // unconditional loads (indices clamped, values masked after): no
        // branch between them and the weight batch, so the first use of x
        // waits for x alone
#pragma unroll
        for (int t = 0; t < kLnMaxT; ++t)
#pragma unroll
            for (int k = 0; k < kLnGroups; ++k) {
                const int e = tid + k * 64 * kSplit;
                const u32x4_t v = ld16(a.x + (int64_t)min(t, a.T - 1) * a.d + min(e, ng - 1) * 8);
                xv[t][k] = t < a.T && e < ng ? v : zero;
            }
#pragma unroll
        for (int k = 0; k < kLnGroups; ++k) {
            const int e = min(tid + k * 64 * kSplit, ng - 1);
            gv[k][0] = *reinterpret_cast<const float4*>(a.gamma + e * 8);
            gv[k][1] = *reinterpret_cast<const float4*>(a.gamma + e * 8 + 4);
        }
        // the first batch (tile indices clamped, so that the loads need no
        // branch; below 64 K tiles the values go unused)
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            wv[u] = ld16_nt(pw + (int64_t)min(w + kSplit * u, KT - 1) * kTileBytes);
#pragma unroll
        for (int t = 0; t < kLnMaxT; ++t) {
            if (t >= a.T) break;
            double sx = 0.0, sq = 0.0;
#pragma unroll
            for (int k = 0; k < kLnGroups; ++k)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const double lo = __uint_as_float(xv[t][k][i] << 16);
                    const double hi = __uint_as_float(xv[t][k][i] & 0xFFFF0000u);
                    sx += lo + hi;
                    sq = fma(lo, lo, fma(hi, hi, sq));
                }
            for (int off = 32; off >= 1; off >>= 1) {
                sx += __shfl_xor(sx, off, 64);
                sq += __shfl_xor(sq, off, 64);
            }
            if (lane == 0) { red[0][t][w] = sx; red[1][t][w] = sq; }
        }
        lds_barrier();
#pragma unroll
        for (int t = 0; t < kLnMaxT; ++t) {
            if (t >= a.T) break;
            double m1 = 0.0, m2 = 0.0;
#pragma unroll
            for (int i = 0; i < kSplit; ++i) { m1 += red[0][t][i]; m2 += red[1][t][i]; }
            const double mean = m1 / a.d;
            const float rstd = (float)(1.0 / sqrt(fmax(m2 / a.d - mean * mean, 0.0) + (double)a.eps));
            const float mu = (float)mean;
#pragma unroll
            for (int k = 0; k < kLnGroups; ++k) {
                const int e = tid + k * 64 * kSplit;
                if (e >= ng) break;
                const float gm[8] = {gv[k][0].x, gv[k][0].y, gv[k][0].z, gv[k][0].w,
                                     gv[k][1].x, gv[k][1].y, gv[k][1].z, gv[k][1].w};
                u32x4_t out;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float lo = (__uint_as_float(xv[t][k][i] << 16) - mu) * rstd * gm[2 * i];
                    const float hi = (__uint_as_float(xv[t][k][i] & 0xFFFF0000u) - mu) * rstd * gm[2 * i + 1];
                    out[i] = (uint32_t)moe::f32_to_bf16(lo) | ((uint32_t)moe::f32_to_bf16(hi) << 16);
                }
                *reinterpret_cast<u32x4_t*>(hs + t * hstride + e * 8) = out;
                if (q == 0) *reinterpret_cast<u32x4_t*>(const_cast<uint16_t*>(a.h) + (int64_t)t * a.d + e * 8) = out;
            }
        }
        lds_barrier();
    }
    // two weight buffers in turn, as gemv_kernel (with kNorm the first batch
    // was issued above, into wv)
    constexpr int kStep = kSplit * kUnroll;
    const int nb = KT / kStep;
    int kt = 0;
    auto xload = [&](int k0, u32x4_t* xv) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int ko = (k0 + w + kSplit * u) * kTileK;
            if constexpr (kNorm) {
                xv[u] = has_tok ? *reinterpret_cast<const u32x4_t*>(hx + ko) : zero;
            } else {
                const u32x4_t v = ld16(px + ko);
                xv[u] = has_tok ? v : zero;
            }
        }
    };
    auto wload = [&](int k0, u32x4_t* wt) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            wt[u] = ld16_nt(pw + (int64_t)(k0 + w + kSplit * u) * kTileBytes);
    };
    auto mfmas = [&](const u32x4_t* wt, const u32x4_t* xv) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc = moe::mfma16x16x32(wt[u], xv[u], acc);
    };
    if (nb > 0) {
        u32x4_t wb[kUnroll];
        if constexpr (!kNorm) wload(0, wv);
        int b = 0;
        for (; b + 2 < nb; b += 2) {
            xload(b * kStep, xb);
            wload((b + 1) * kStep, wb);
            mfmas(wv, xb);
            xload((b + 1) * kStep, xb);
            wload((b + 2) * kStep, wv);
            mfmas(wb, xb);
        }
        xload(b * kStep, xb);
        if (b + 1 < nb) {
            wload((b + 1) * kStep, wb);
            mfmas(wv, xb);
            xload((b + 1) * kStep, xb);
            mfmas(wb, xb);
        } else {
            mfmas(wv, xb);
        }
        kt = nb * kStep;
    }
    for (kt += w; kt < KT; kt += kSplit) {
        const u32x4_t wt = ld16_nt(pw + (int64_t)kt * kTileBytes);
        u32x4_t xt;
        if constexpr (kNorm)
            xt = has_tok ? *reinterpret_cast<const u32x4_t*>(hx + kt * kTileK) : zero;
        else
            xt = has_tok ? ld16(px + kt * kTileK) : zero;
        acc = moe::mfma16x16x32(wt, xt, acc);
    }
    if (w > 0) s_red[(w - 1) * 64 + lane] = acc;
    __syncthreads();
    if (w != 0) return;
    for (int i = 0; i + 1 < kSplit; ++i) acc += s_red[i * 64 + lane];
    if (!has_tok) return;
    const int hd = a.hd, half = hd / 2;
    const int nqk = (a.H + a.G) * hd, nqkv = nqk + a.G * hd;
    const int row0 = q * kTileRows;
    const int pos = a.pos0 + j;
    float* qrow = a.qkv + (int64_t)j * nqkv;
    uint16_t* dst;
    float r[4];
    if (row0 < nqk) {
        const int head = row0 / hd, m = (row0 % hd) / kTileRows;
        const bool second = g >= 2;
        const int f0 = 8 * m + 4 * (g & 1);           // frequency index of acc[0]
        const int i0 = (second ? half : 0) + f0;       // feature index in the head
        *reinterpret_cast<float4*>(qrow + head * hd + i0) = make_float4(acc[0], acc[1], acc[2], acc[3]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float partner = __shfl_xor(acc[e], 32, 64);
            float c, sf;
            rope_cs(pos, a.inv_freq[f0 + e], c, sf);
            r[e] = second ? acc[e] * c + partner * sf : acc[e] * c - partner * sf;
        }
        dst = head < a.H ? a.q + ((int64_t)j * a.H + head) * hd + i0
                         : a.kc + ((int64_t)(head - a.H) * a.max_seq + pos) * hd + i0;
    } else {
        const int n = row0 + 4 * g;                    // value features: natural order
        *reinterpret_cast<float4*>(qrow + n) = make_float4(acc[0], acc[1], acc[2], acc[3]);
#pragma unroll
        for (int e = 0; e < 4; ++e) r[e] = acc[e];
        dst = a.vc + ((int64_t)((n - nqk) / hd) * a.max_seq + pos) * hd + (n - nqk) % hd;
    }
    const uint32_t lo = (uint32_t)moe::f32_to_bf16(r[0]) | ((uint32_t)moe::f32_to_bf16(r[1]) << 16);
    const uint32_t hi = (uint32_t)moe::f32_to_bf16(r[2]) | ((uint32_t)moe::f32_to_bf16(r[3]) << 16);
    *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
}

struct ScoreArgs {
    const uint16_t* q;     // [T][H][hd] bf16
    const uint16_t* kc;    // [G][max_seq][hd]
    const uint16_t* vc;
    float* part;           // [T][H][n_chunks][hd + kPartPad]: sum of p v, then m, l
    int T, H, G, max_seq, pos0, n_chunks;
    float scale;           // 1 / sqrt(hd)
};

// One workgroup of 4 waves per (key/value head g, chunk c of 64 positions);
// wave w owns positions 16 w .. 16 w + 15 of the chunk.  The query rows are
// every (token t, query head j of g), r = t * group + jj, in batches of 16;
// row r sees positions up to pos0 + t (causal).
//
// Scores on the matrix cores: v_mfma_f32_16x16x32_bf16 with the wave's 16
// positions x 32 dims of K as the A operand (lane l: position l%16, dims
// 8(l/16)..+7) and the batch's q rows as B, so lane l ends with the scores of
// query row l%16 at positions 16 w + 4(l/16) + i (i = 0..3).  The chunk's
// maximum per row is the maximum of the four waves' (two butterfly steps in
// the wave, then LDS), exp(s - max) goes to LDS and the chunk's sum adds the
// waves' sums in wave order.  Then wave w sums P v over all 64 positions for
// dims w hd/4 .. (w+1) hd/4 - 1: lane l takes dims D(l%16)..+D-1 of that
// quarter at positions 4k + l/16 (V staged in LDS, rows padded so the four
// position groups hit distinct banks), two butterfly steps adding the four
// position groups in a fixed order.
template <int HD>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a)
{
    constexpr int kPos = 64;           // positions per workgroup
    constexpr int kWaves = 4;          // 16 positions per wave
    constexpr int KS = HD / 32;        // MFMA K steps over the head
    constexpr int DQ = HD / kWaves;    // dims per wave in P v
    constexpr int D = DQ / 16;         // dims per lane in P v
    constexpr int VROW = HD + 32;      // padded V row (bf16)
    __shared__ __attribute__((aligned(16))) uint16_t vs[kPos * VROW];
    __shared__ float ps[16][kPos + 4];
    __shared__ float mx[kWaves][16], lx[kWaves][16];
    const int g = blockIdx.x, c = blockIdx.y;
    const int group = a.H / a.G;
    const int R = a.T * group;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int p0 = c * kPos;
    const int n_pos = a.pos0 + a.T;
    const int last = min(kPos, n_pos - p0);          // live positions of the chunk
    const uint16_t* kbase = a.kc + (int64_t)g * a.max_seq * HD;
    const uint16_t* vbase = a.vc + (int64_t)g * a.max_seq * HD;
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    // K fragments of the wave's 16 positions (A operands), loaded once
    u32x4_t kf[KS];
    {
        const int p = w * 16 + (lane & 15);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            kf[ks] = p < last ? ld16(kbase + (int64_t)(p0 + p) * HD + ks * 32 + (lane >> 4) * 8)
                              : zero;
    }
    // V of the wave's 16 positions into LDS (16-byte pieces, coalesced)
    for (int e = lane; e < 16 * (HD / 8); e += 64) {
        const int p = w * 16 + e / (HD / 8), k8 = e % (HD / 8);
        *reinterpret_cast<u32x4_t*>(&vs[p * VROW + k8 * 8]) =
            p < last ? ld16(vbase + (int64_t)(p0 + p) * HD + k8 * 8) : zero;
    }
    const int dg = lane & 15, pq = lane >> 4;
    for (int b0 = 0; b0 < R; b0 += 16) {
        const int c_row = b0 + dg;                      // this lane's query row
        const bool row_ok = c_row < R;
        const int t_row = row_ok ? c_row / group : 0;
        const int j_row = g * group + (row_ok ? c_row % group : 0);
        const uint16_t* qrow = a.q + ((int64_t)t_row * a.H + j_row) * HD + pq * 8;
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const u32x4_t qb = row_ok ? ld16(qrow + ks * 32) : zero;
            acc = moe::mfma16x16x32(kf[ks], qb, acc);
        }
        // scale, causal mask, the chunk's maximum per row
        const int lim = a.pos0 + t_row;
        float sv[4];
        float m = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int pos = p0 + w * 16 + pq * 4 + i;
            sv[i] = (row_ok && pos <= lim) ? acc[i] * a.scale : -INFINITY;
            m = fmaxf(m, sv[i]);
        }
        m = fmaxf(m, __shfl_xor(m, 16, 64));
        m = fmaxf(m, __shfl_xor(m, 32, 64));
        if (lane < 16) mx[w][lane] = m;
        __syncthreads();
        m = fmaxf(fmaxf(mx[0][dg], mx[1][dg]), fmaxf(mx[2][dg], mx[3][dg]));
        float l = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float p = sv[i] == -INFINITY ? 0.f : expf(sv[i] - m);
            l += p;
            ps[dg][w * 16 + pq * 4 + i] = p;
        }
        l += __shfl_xor(l, 16, 64);
        l += __shfl_xor(l, 32, 64);
        if (lane < 16) lx[w][lane] = l;
        __syncthreads();
        // row statistics of the chunk: wave 0, lanes of the first position group
        if (w == 0 && pq == 0 && row_ok) {
            float* out = a.part + (((int64_t)t_row * a.H + j_row) * a.n_chunks + c) * (HD + kPartPad);
            out[HD] = m;
            out[HD + 1] = ((lx[0][dg] + lx[1][dg]) + lx[2][dg]) + lx[3][dg];
        }
        // P v for this wave's quarter of the dims, 8 rows at a time
        const int nb = min(16, R - b0);
        for (int r0 = 0; r0 < nb; r0 += 8) {
            float o[8][D];
#pragma unroll
            for (int rr = 0; rr < 8; ++rr)
#pragma unroll
                for (int e = 0; e < D; ++e) o[rr][e] = 0.f;
#pragma unroll 4
            for (int k = 0; k < kPos / 4; ++k) {
                const int p = 4 * k + pq;
                const uint16_t* vr = &vs[p * VROW + w * DQ + dg * D];
                float vv[D];
                if constexpr (D == 2) {
                    const uint32_t w2 = *reinterpret_cast<const uint32_t*>(vr);
                    vv[0] = __uint_as_float(w2 << 16);
                    vv[1] = __uint_as_float(w2 & 0xFFFF0000u);
                } else {
                    vv[0] = __uint_as_float((uint32_t)vr[0] << 16);
                }
#pragma unroll
                for (int rr = 0; rr < 8; ++rr) {
                    const float pw = ps[r0 + rr][p];
#pragma unroll
                    for (int e = 0; e < D; ++e) o[rr][e] = fmaf(pw, vv[e], o[rr][e]);
                }
            }
#pragma unroll
            for (int rr = 0; rr < 8; ++rr)
#pragma unroll
                for (int e = 0; e < D; ++e) {
                    float v = o[rr][e];
                    v += __shfl_xor(v, 16, 64);
                    v += __shfl_xor(v, 32, 64);
                    o[rr][e] = v;
                }
            if (pq == 0) {
#pragma unroll
                for (int rr = 0; rr < 8; ++rr) {
                    const int r = b0 + r0 + rr;
                    if (r < R) {
                        const int t = r / group, j = g * group + r % group;
                        float* out = a.part + (((int64_t)t * a.H + j) * a.n_chunks + c) * (HD + kPartPad);
#pragma unroll
                        for (int e = 0; e < D; ++e) out[w * DQ + dg * D + e] = o[rr][e];
                    }
                }
            }
        }
        __syncthreads();
    }
}

struct CombineArgs {
    const float* part;
    uint16_t* out;         // [T][H * hd] bf16
    int H, hd, pos0, n_chunks;
};

// (token t, head j) per workgroup, one thread per dimension: the chunks that
// hold positions of t, merged by their maxima in chunk order
__global__ __launch_bounds__(128) void combine_kernel(CombineArgs a)
{
    const int th = blockIdx.x, t = th / a.H;
    const int i = threadIdx.x;
    if (i >= a.hd) return;
    const int used = (a.pos0 + t) / kChunk + 1;
    const int stride = a.hd + kPartPad;
    const float* base = a.part + (int64_t)th * a.n_chunks * stride;
    float M = -INFINITY;
#pragma unroll 8
    for (int c = 0; c < used; ++c) M = fmaxf(M, base[(int64_t)c * stride + a.hd]);
    float L = 0.f, acc = 0.f;
#pragma unroll 8
    for (int c = 0; c < used; ++c) {
        const float* pc = base + (int64_t)c * stride;
        const float f = expf(pc[a.hd] - M);
        L = fmaf(pc[a.hd + 1], f, L);
        acc = fmaf(pc[i], f, acc);
    }
    a.out[(int64_t)th * a.hd + i] = moe::f32_to_bf16(acc / L);
}

// ---------------------------------------------------------------- prefill
// More than 16 new tokens: the projections run on the grouped GEMM of
// moe_prefill.hip (one "expert", its rows the tokens), then these kernels.

// rope_kernel, one workgroup per token: from the projection's fp32 output
// in packed row order (query and key features placed by rope_row), the
// natural-order fp32 q|k|v (kept for inspection), q rotated to bf16 in the
// workspace, k rotated and v to the cache at position pos0 + t.  The angle
// and rotation arithmetic are the decode epilogue's (rope_cs).
struct RopeArgs {
    const float* qkvp;     // [T][nqkv] fp32, packed row order
    const double* inv_freq;
    float* qkv;            // [T][nqkv] fp32, natural order
    uint16_t* q;           // [T][H][hd]
    uint16_t* kc;
    uint16_t* vc;
    int T, H, G, hd, max_seq, pos0;
};

__global__ __launch_bounds__(256) void rope_kernel(RopeArgs a)
{
    const int t = blockIdx.x;
    const int hd = a.hd, half = hd / 2;
    const int nqk = (a.H + a.G) * hd, nqkv = nqk + a.G * hd;
    const int pos = a.pos0 + t;
    const float* src = a.qkvp + (int64_t)t * nqkv;
    float* nat = a.qkv + (int64_t)t * nqkv;
    for (int e = threadIdx.x; e < (a.H + a.G) * half; e += blockDim.x) {
        const int head = e / half, f = e % half;
        const int n0 = head * hd + f, n1 = n0 + half;
        const float x0 = src[moe::rope_row(n0, hd)], x1 = src[moe::rope_row(n1, hd)];
        nat[n0] = x0;
        nat[n1] = x1;
        float c, sf;
        rope_cs(pos, a.inv_freq[f], c, sf);
        const float r0 = x0 * c - x1 * sf, r1 = x1 * c + x0 * sf;
        uint16_t* dst = head < a.H ? a.q + ((int64_t)t * a.H + head) * hd
                                   : a.kc + ((int64_t)(head - a.H) * a.max_seq + pos) * hd;
        dst[f] = moe::f32_to_bf16(r0);
        dst[f + half] = moe::f32_to_bf16(r1);
    }
    for (int e = threadIdx.x; e < a.G * hd; e += blockDim.x) {
        const float v = src[nqk + e];
        nat[nqk + e] = v;
        a.vc[((int64_t)(e / hd) * a.max_seq + pos) * hd + e % hd] = moe::f32_to_bf16(v);
    }
}

// flash_kernel: causal attention of T new tokens, one workgroup of 4 waves
// per (query head j, block of 128 query tokens); wave w owns tokens
// 32 w .. 32 w + 31 of the block, one per lane column (lanes l and l + 32
// share token l % 32).  Per step of 64 positions of head j's key/value head:
// K rows and V transposed (dims major) go to LDS; the scores are computed
// transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16 (A = 32 positions x
// 16 dims of K from LDS, B = the wave's query rows), so lane l ends with the
// scores of token l % 32 at positions 8 g + 4 (l / 32) + r of each
// 32-position block (register 4 g + r); the running maximum and sum per
// token (one exchange between the lane pair) rescale the output, and
// O^T += V^T P^T takes the P values straight from those registers as the B
// operand: the 16-position K step s of a block takes registers g = 2 s,
// 2 s + 1, i.e. positions 16 s + {4 h .. 4 h + 3, 8 + 4 h .. 8 + 4 h + 3}
// for h = l / 32, and the V^T operand is read from LDS in the same order.
// P enters the matrix cores as two bf16 terms, bf16(p) and bf16(p - bf16(p)),
// which keep 16 significant bits; V is bf16 and every product is exact in
// the fp32 accumulation.
struct FlashArgs {
    const uint16_t* q;     // [T][H][HD] bf16, rotated
    const uint16_t* kc;    // this layer's K cache [G][max_seq][HD]
    const uint16_t* vc;
    uint16_t* out;         // a [T][H * HD] bf16
    int T, H, G, max_seq, pos0;
    int nqb;               // query blocks of kFlashQ tokens
    float scale2;          // 1/sqrt(head_dim) * log2(e): scores in base 2
};

constexpr int kXcds = 8;

constexpr int kFlashQ = 128;    // query tokens per workgroup
constexpr int kFlashP = 64;     // positions per step

__device__ inline uint32_t pack_bf16x2(float lo, float hi)
{
    return (uint32_t)moe::f32_to_bf16(lo) | ((uint32_t)moe::f32_to_bf16(hi) << 16);
}

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

__device__ inline f32x16_t mfma32x32x16(const u32x4_t a, const u32x4_t b, f32x16_t c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(moe::bf16x8_t, a),
                                                   __builtin_bit_cast(moe::bf16x8_t, b), c, 0, 0, 0);
}

// Two workgroups per CU: 219 registers per lane at head_dim 128 (the output
// block of 32 tokens x 128 dims alone takes 64), 2 waves per SIMD.
template <int HD>
__global__ __launch_bounds__(256, 2) void flash_kernel(FlashArgs a)
{
    constexpr int KQ = HD / 16;              // 16-dim K steps of the score MFMAs
    constexpr int DB = HD / 32;              // 32-dim blocks of the output
    constexpr int KROW = HD + 8;             // padded K row in LDS (bf16)
    // padded V^T row (positions, bf16): 34 words, so the 8-byte reads of
    // consecutive dims fall in distinct bank pairs (LDS bank conflicts 19.5 M
    // -> 6.5 M cycles per launch against 36 words)
    constexpr int VROW = kFlashP + 4;
    __shared__ __attribute__((aligned(16))) uint16_t ks[kFlashP * KROW];
    __shared__ __attribute__((aligned(16))) uint16_t vt[HD * VROW];
    // XCD-aware numbering: hardware hands block b to XCD b % 8, and each XCD
    // takes a contiguous run of the logical order (key/value head, query
    // block from the last, query head of the group), so the workgroups of
    // one key/value head share its K and V in one L2 (DBRX: one head per
    // XCD) and on every XCD the longest query blocks (the most positions)
    // start first.  Logical slots past the last block exit at once.
    const int groups = a.H / a.G;
    const int per_xcd = gridDim.x / kXcds;
    const int logical = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (logical >= a.H * a.nqb) return;
    const int kvh = logical / (a.nqb * groups), rem = logical % (a.nqb * groups);
    const int qb = a.nqb - 1 - rem / groups;
    const int j = kvh * groups + rem % groups;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = lane & 31, h = lane >> 5;
    const int t_w0 = qb * kFlashQ + w * 32;             // the wave's first token
    const int t = t_w0 + c;                              // this lane's token
    const bool tok_ok = t < a.T;
    const int lim = a.pos0 + t;                          // its last position
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    u32x4_t qf[KQ];
    {
        const uint16_t* qrow = a.q + ((int64_t)(tok_ok ? t : 0) * a.H + j) * HD + h * 8;
#pragma unroll
        for (int k = 0; k < KQ; ++k) {
            const u32x4_t v = ld16(qrow + k * 16);
            qf[k] = tok_ok ? v : zero;
        }
    }
    f32x16_t o[DB];
#pragma unroll
    for (int b = 0; b < DB; ++b) o[b] = f32x16_t{};
    float m = -INFINITY, l = 0.f;
    const int t_last = min(qb * kFlashQ + kFlashQ, a.T) - 1;
    const int n_pos = a.pos0 + t_last + 1;               // positions the block needs
    const uint16_t* kbase = a.kc + (int64_t)kvh * a.max_seq * HD;
    const uint16_t* vbase = a.vc + (int64_t)kvh * a.max_seq * HD;
    uint32_t* vt32 = reinterpret_cast<uint32_t*>(vt);
    // per step a thread stages KL 16-byte pieces of K rows and VL position
    // pairs of V; all of a step's global loads are issued before the barrier
    // that frees the LDS, so the step waits for one load latency, not one per
    // piece
    constexpr int KL = kFlashP * (HD / 8) / 256;
    constexpr int VL = (kFlashP / 2) * (HD / 8) / 256;
    static_assert(KL * 256 == kFlashP * (HD / 8) && VL * 256 == (kFlashP / 2) * (HD / 8),
                  "the staging pieces divide evenly over the 256 threads");
    for (int p0 = 0; p0 < n_pos; p0 += kFlashP) {
        const int live = min(kFlashP, n_pos - p0);
        u32x4_t kv[KL], va[VL], vb[VL];
#pragma unroll
        for (int i = 0; i < KL; ++i) {
            const int e = threadIdx.x + i * 256;
            const int p = e / (HD / 8), k8 = e % (HD / 8);
            kv[i] = ld16(kbase + (int64_t)(p0 + min(p, live - 1)) * HD + k8 * 8);
        }
#pragma unroll
        for (int i = 0; i < VL; ++i) {
            const int e = threadIdx.x + i * 256;
            const int pp = e % (kFlashP / 2), k8 = e / (kFlashP / 2);
            va[i] = ld16(vbase + (int64_t)(p0 + min(2 * pp, live - 1)) * HD + k8 * 8);
            vb[i] = ld16(vbase + (int64_t)(p0 + min(2 * pp + 1, live - 1)) * HD + k8 * 8);
        }
        __syncthreads();                                 // the last step's LDS reads are done
        // K rows: 16-byte pieces, coalesced.  Rows past `live` repeat the
        // last live row (the loads are clamped): every token's causal mask
        // removes those positions, so their scores never count and their
        // probabilities are exactly 0 against finite V rows.
#pragma unroll
        for (int i = 0; i < KL; ++i) {
            const int e = threadIdx.x + i * 256;
            const int p = e / (HD / 8), k8 = e % (HD / 8);
            *reinterpret_cast<u32x4_t*>(&ks[p * KROW + k8 * 8]) = kv[i];
        }
        // V transposed: a thread takes positions 2 pp, 2 pp + 1 at 8 dims and
        // writes 8 words of (position pair) per dim, each one byte permute
        // (low halves of the two words, then the high halves)
#pragma unroll
        for (int i = 0; i < VL; ++i) {
            const int e = threadIdx.x + i * 256;
            const int pp = e % (kFlashP / 2), k8 = e / (kFlashP / 2);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                vt32[((k8 * 8 + 2 * r) * VROW) / 2 + pp] = __builtin_amdgcn_perm(vb[i][r], va[i][r], 0x05040100u);
                vt32[((k8 * 8 + 2 * r + 1) * VROW) / 2 + pp] = __builtin_amdgcn_perm(vb[i][r], va[i][r], 0x07060302u);
            }
        }
        __syncthreads();
        // S^T = K Q^T for the two 32-position blocks: lane (c, h) ends with
        // token c's scores at positions 32 pb + 8 g + 4 h + r (register 4 g + r)
        f32x16_t st[2];
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
            st[pb] = f32x16_t{};
#pragma unroll
            for (int k = 0; k < KQ; ++k) {
                const u32x4_t kf =
                    *reinterpret_cast<const u32x4_t*>(&ks[(pb * 32 + c) * KROW + k * 16 + h * 8]);
                st[pb] = mfma32x32x16(kf, qf[k], st[pb]);
            }
        }
        // scores in base 2 (s * scale * log2 e, so p = 2^(s2 - m2)); the
        // causal mask and the tokens past T only on the steps that need them
        // (wave-uniform: a step past the wave's first token's last position,
        // or a wave with tokens past T)
        float sv[32];
        float mx = -INFINITY;
        if (p0 + kFlashP - 1 > a.pos0 + t_w0 || t_w0 + 31 >= a.T) {
#pragma unroll
            for (int pb = 0; pb < 2; ++pb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int pos = p0 + pb * 32 + 8 * (i / 4) + 4 * h + (i % 4);
                    const float v = (tok_ok && pos <= lim) ? st[pb][i] * a.scale2 : -INFINITY;
                    sv[pb * 16 + i] = v;
                    mx = fmaxf(mx, v);
                }
        } else {
#pragma unroll
            for (int pb = 0; pb < 2; ++pb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    sv[pb * 16 + i] = st[pb][i] * a.scale2;
                    mx = fmaxf(mx, sv[pb * 16 + i]);
                }
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float mn = fmaxf(m, mx);
        // a token with every position masked so far (only tokens past T)
        // keeps mn = -inf: subtract 0 instead, so its p are 0, not NaN
        const float msub = mn == -INFINITY ? 0.f : mn;
        float ps = 0.f;
        float pv[32];
#pragma unroll
        for (int e = 0; e < 32; ++e) {
            pv[e] = __builtin_amdgcn_exp2f(sv[e] - msub);
            ps += pv[e];
        }
        ps += __shfl_xor(ps, 32, 64);
        // rescale the running sums only where a maximum moved (m == mn gives
        // the factor 1 exactly, so skipping it changes no bit)
        if (__ballot(mn != m)) {
            const float alpha = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mn);
            l *= alpha;
#pragma unroll
            for (int b = 0; b < DB; ++b) o[b] *= alpha;
        }
        l += ps;
        m = mn;
        // O^T += V^T P^T, four 16-position K steps: step (pb, s) takes the
        // lane's registers 4 g + r for g = 2 s, 2 s + 1 of block pb, i.e.
        // positions 32 pb + 16 s + {4 h .. 4 h + 3, 8 + 4 h .. 8 + 4 h + 3},
        // and the V^T operand is read in the same order; P as hi + lo,
        // hi = bf16(p), lo = bf16(p - hi) (the subtraction is exact)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
            for (int sx = 0; sx < 2; ++sx) {
                const float* pp = &pv[pb * 16 + sx * 8];
                u32x4_t bh, bl;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t hw = moe::cvt_pk_bf16(pp[2 * i], pp[2 * i + 1]);
                    bh[i] = hw;
                    bl[i] = moe::cvt_pk_bf16(pp[2 * i] - __uint_as_float(hw << 16),
                                             pp[2 * i + 1] - __uint_as_float(hw & 0xFFFF0000u));
                }
#pragma unroll
                for (int b = 0; b < DB; ++b) {
                    const uint32_t* vr = vt32 + ((b * 32 + c) * VROW + pb * 32 + sx * 16 + 4 * h) / 2;
                    const uint2 v0 = *reinterpret_cast<const uint2*>(vr);
                    const uint2 v1 = *reinterpret_cast<const uint2*>(vr + 4);
                    const u32x4_t av = {v0.x, v0.y, v1.x, v1.y};
                    o[b] = mfma32x32x16(av, bh, o[b]);
                    o[b] = mfma32x32x16(av, bl, o[b]);
                }
            }
    }
    if (!tok_ok) return;
    // lane: dims 32 b + 8 g + 4 h + r of token t (register 4 g + r)
    const float inv = 1.0f / l;
    uint16_t* dst = a.out + ((int64_t)t * a.H + j) * HD + 4 * h;
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int g = 0; g < 4; ++g)
            *reinterpret_cast<uint2*>(dst + b * 32 + 8 * g) =
                make_uint2(pack_bf16x2(o[b][4 * g] * inv, o[b][4 * g + 1] * inv),
                           pack_bf16x2(o[b][4 * g + 2] * inv, o[b][4 * g + 3] * inv));
}

// y = bf16(x + o), 8 elements per thread
__global__ __launch_bounds__(256) void residual_kernel(const uint16_t* __restrict__ x,
                                                       const float* __restrict__ o,
                                                       uint16_t* y, int64_t n8)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n8) return;
    const u32x4_t xv = ld16(x + i * 8);
    const float4 o0 = *reinterpret_cast<const float4*>(o + i * 8);
    const float4 o1 = *reinterpret_cast<const float4*>(o + i * 8 + 4);
    const float ov[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
    u32x4_t out;
#pragma unroll
    for (int k = 0; k < 4; ++k)
        out[k] = pack_bf16x2(__uint_as_float(xv[k] << 16) + ov[2 * k],
                             __uint_as_float(xv[k] & 0xFFFF0000u) + ov[2 * k + 1]);
    *reinterpret_cast<u32x4_t*>(y + i * 8) = out;
}

}  // namespace attn

extern "C" {

hipError_t attn_launch_norm(const uint16_t* x, const float* gamma, int T, int d, float eps,
                            uint16_t* h, hipStream_t s)
{
    hipLaunchKernelGGL(attn::norm_kernel, dim3(T), dim3(attn::kNormThreads), 0, s, x, gamma, d,
                       eps, h);
    return hipGetLastError();
}

int attn_norm_in_projection(int T) { return T <= attn::kLnMaxT; }

hipError_t attn_launch_qkv(const void* w, uint16_t* h, const uint16_t* x, const float* gamma,
                           float eps, const double* inv_freq, float* qkv, uint16_t* q,
                           uint16_t* kc, uint16_t* vc, int T, int d, int H, int G, int hd,
                           int max_seq, int pos0, hipStream_t s)
{
    attn::QkvArgs a{static_cast<const uint8_t*>(w), h, x, gamma, eps, inv_freq, qkv, q, kc, vc,
                    d, T, H, G, hd, max_seq, pos0};
    const int rows = (H + 2 * G) * hd;
    const dim3 grid(rows / moe::kTileRows), block(64 * attn::kSplit);
    if (attn_norm_in_projection(T)) {
        const size_t lds = (size_t)T * (d + attn::kHPad) * 2;
        hipLaunchKernelGGL(attn::qkv_kernel<true>, grid, block, lds, s, a);
    } else {
        hipLaunchKernelGGL(attn::qkv_kernel<false>, grid, block, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t attn_launch_out(const void* w, const uint16_t* x, int T, int K, int N, float* y32,
                           const uint16_t* res, uint16_t* y16, hipStream_t s)
{
    attn::GemvArgs a{static_cast<const uint8_t*>(w), x, y32, res, y16, K, N, T};
    hipLaunchKernelGGL(attn::gemv_kernel, dim3(N / moe::kTileRows), dim3(64 * attn::kSplit), 0, s, a);
    return hipGetLastError();
}

int attn_chunks(int n_pos) { return (n_pos + attn::kChunk - 1) / attn::kChunk; }
int attn_part_stride(int hd) { return hd + attn::kPartPad; }

hipError_t attn_launch_score(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                             float* part, int T, int H, int G, int hd, int max_seq, int pos0,
                             int n_chunks_alloc, hipStream_t s)
{
    const int n_chunks = attn_chunks(pos0 + T);
    attn::ScoreArgs a{q, kc, vc, part, T, H, G, max_seq, pos0, n_chunks_alloc,
                      (float)(1.0 / sqrt((double)hd))};
    if (hd == 128)
        hipLaunchKernelGGL(attn::score_kernel<128>, dim3(G, n_chunks), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(attn::score_kernel<64>, dim3(G, n_chunks), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t attn_launch_rope(const float* qkvp, const double* inv_freq, float* qkv, uint16_t* q,
                            uint16_t* kc, uint16_t* vc, int T, int H, int G, int hd, int max_seq,
                            int pos0, hipStream_t s)
{
    attn::RopeArgs a{qkvp, inv_freq, qkv, q, kc, vc, T, H, G, hd, max_seq, pos0};
    hipLaunchKernelGGL(attn::rope_kernel, dim3(T), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t attn_launch_flash(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                             uint16_t* out, int T, int H, int G, int hd, int max_seq, int pos0,
                             hipStream_t s)
{
    const int nqb = (T + attn::kFlashQ - 1) / attn::kFlashQ;
    attn::FlashArgs a{q, kc, vc, out, T, H, G, max_seq, pos0, nqb,
                      (float)(1.4426950408889634 / sqrt((double)hd))};
    const dim3 grid((H * nqb + attn::kXcds - 1) / attn::kXcds * attn::kXcds);
    if (hd == 128)
        hipLaunchKernelGGL(attn::flash_kernel<128>, grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(attn::flash_kernel<64>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t attn_launch_residual(const uint16_t* x, const float* o, uint16_t* y, int64_t n,
                                hipStream_t s)
{
    const int64_t n8 = n / 8;
    hipLaunchKernelGGL(attn::residual_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, s,
                       x, o, y, n8);
    return hipGetLastError();
}

hipError_t attn_launch_combine(const float* part, uint16_t* out, int T, int H, int hd, int pos0,
                               int n_chunks_alloc, hipStream_t s)
{
    attn::CombineArgs c{part, out, H, hd, pos0, n_chunks_alloc};
    hipLaunchKernelGGL(attn::combine_kernel, dim3(T * H), dim3(128), 0, s, c);
    return hipGetLastError();
}

}  // extern "C"
