// attn.hip -- kernels of the self-attention block of include/attn.h for a few
// new tokens (T <= 16: decode), in launch order:
//
//   norm_kernel     layer norm of x, one workgroup per token (fp32 statistics,
//                   fixed reduction order), h = bf16((x - mean) rstd gamma)
//   gemv_kernel<kQkv>  q|k|v = h Wqkv, fp32
//   rope_kernel     rotary encoding of the query and key heads (angles in
//                   fp64, rotation in fp32), bf16 q to the workspace, bf16 k
//                   and v appended to the cache
//   score_kernel    attention of every query head of one key/value head over
//                   one chunk of 256 positions: scores, the chunk's softmax
//                   maximum and sum, and the unnormalised weighted sum of v
//   combine_kernel  merges the chunks of each (token, head) into bf16 a
//   gemv_kernel<kOut>  o = a Wo (fp32) and y = bf16(x + o)
//
// The GEMVs stream the fragment-tiled weights (the layout of moe_common.h)
// through v_mfma_f32_16x16x32_bf16 with the tokens as the B operand, as the
// MoE decode GEMVs do: one workgroup per 16 output features, its 8 waves
// splitting K (wave w takes K tiles w, w + 8, ...), wave 0 adding the
// partial fragments in wave order.  The attention is VALU work: per token
// and head it is q . k over hd for each position and a weighted sum of v,
// small beside the projections' weight stream.
#include "moe_common.h"

namespace attn {

using moe::f32x4_t;
using moe::u32x4_t;
using moe::kTileK;
using moe::kTileBytes;
using moe::kTileRows;

constexpr int kNormThreads = 256;
constexpr int kSplit = 8;          // waves per GEMV workgroup (K split)
constexpr int kUnroll = 8;         // K tiles per wave in flight
constexpr int kChunk = 256;        // positions per attention workgroup (one per thread)
constexpr int kRowBatch = 16;      // query rows whose P is held in LDS at once
constexpr int kMaxRows = 16 * 8;   // tokens (16) x query heads per key/value head (8)
constexpr int kPartPad = 4;        // m, l and padding after the hd sums of a partial

__device__ inline u32x4_t ld16_nt(const void* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}

__device__ inline u32x4_t ld16(const void* p) { return *reinterpret_cast<const u32x4_t*>(p); }

// sum over the 256 threads of a workgroup: lane butterfly, then the 4 wave
// sums in wave order (the same order every time)
__device__ inline float block_sum(float v, float* red)
{
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    return ((red[0] + red[1]) + red[2]) + red[3];
}

__global__ __launch_bounds__(kNormThreads) void norm_kernel(const uint16_t* __restrict__ x,
                                                            const float* __restrict__ gamma,
                                                            int d, float eps,
                                                            uint16_t* __restrict__ h)
{
    __shared__ float red[4];
    const int t = blockIdx.x;
    const uint16_t* xr = x + (int64_t)t * d;
    // thread i holds the 8-element groups i, i + 256, ... (d % 256 == 0)
    float s = 0.f;
    for (int g = threadIdx.x; g < d / 8; g += kNormThreads) {
        const u32x4_t v = ld16(xr + g * 8);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            s += __uint_as_float(v[k] << 16) + __uint_as_float(v[k] & 0xFFFF0000u);
    }
    const float mean = block_sum(s, red) / (float)d;
    float q = 0.f;
    for (int g = threadIdx.x; g < d / 8; g += kNormThreads) {
        const u32x4_t v = ld16(xr + g * 8);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float a = __uint_as_float(v[k] << 16) - mean;
            const float b = __uint_as_float(v[k] & 0xFFFF0000u) - mean;
            q = fmaf(a, a, q);
            q = fmaf(b, b, q);
        }
    }
    const float var = block_sum(q, red) / (float)d;
    const float rstd = 1.0f / sqrtf(var + eps);
    for (int g = threadIdx.x; g < d / 8; g += kNormThreads) {
        const u32x4_t v = ld16(xr + g * 8);
        const float4 g0 = *reinterpret_cast<const float4*>(gamma + g * 8);
        const float4 g1 = *reinterpret_cast<const float4*>(gamma + g * 8 + 4);
        const float gm[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        u32x4_t out;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float a = (__uint_as_float(v[k] << 16) - mean) * rstd * gm[2 * k];
            const float b = (__uint_as_float(v[k] & 0xFFFF0000u) - mean) * rstd * gm[2 * k + 1];
            out[k] = (uint32_t)moe::f32_to_bf16(a) | ((uint32_t)moe::f32_to_bf16(b) << 16);
        }
        *reinterpret_cast<u32x4_t*>(h + (int64_t)t * d + g * 8) = out;
    }
}

enum { kQkv = 0, kOut = 1 };

struct GemvArgs {
    const uint8_t* w;      // packed weights: N/16 row tiles of K/32 tiles
    const uint16_t* x;     // [T][K] bf16
    float* y32;            // [T][N] fp32
    const uint16_t* res;   // kOut: residual [T][N] bf16
    uint16_t* y16;         // kOut: bf16(res + y) [T][N]
    int K, N, T;
};

template <int kMode>
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
    int kt = 0;
    for (; kt + kSplit * kUnroll <= KT; kt += kSplit * kUnroll) {
        u32x4_t wv[kUnroll], xb[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            wv[u] = ld16_nt(pw + (int64_t)(kt + w + kSplit * u) * kTileBytes);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            xb[u] = has_tok ? ld16(px + (kt + w + kSplit * u) * kTileK) : zero;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc = moe::mfma16x16x32(wv[u], xb[u], acc);
    }
    for (kt += w; kt < KT; kt += kSplit) {
        const u32x4_t wv = ld16_nt(pw + (int64_t)kt * kTileBytes);
        const u32x4_t xb = has_tok ? ld16(px + kt * kTileK) : zero;
        acc = moe::mfma16x16x32(wv, xb, acc);
    }
    if (w > 0) s_red[(w - 1) * 64 + lane] = acc;
    __syncthreads();
    if (w != 0) return;
    for (int i = 0; i + 1 < kSplit; ++i) acc += s_red[i * 64 + lane];
    if (!has_tok) return;
    // lane holds output features 16q + 4g .. +3 of token j
    const int64_t o = (int64_t)j * a.N + q * kTileRows + g * 4;
    *reinterpret_cast<float4*>(a.y32 + o) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    if (kMode == kOut) {
        const uint2 r = *reinterpret_cast<const uint2*>(a.res + o);
        const float r0 = __uint_as_float(r.x << 16), r1 = __uint_as_float(r.x & 0xFFFF0000u);
        const float r2 = __uint_as_float(r.y << 16), r3 = __uint_as_float(r.y & 0xFFFF0000u);
        const uint32_t lo = (uint32_t)moe::f32_to_bf16(r0 + acc[0]) |
                            ((uint32_t)moe::f32_to_bf16(r1 + acc[1]) << 16);
        const uint32_t hi = (uint32_t)moe::f32_to_bf16(r2 + acc[2]) |
                            ((uint32_t)moe::f32_to_bf16(r3 + acc[3]) << 16);
        *reinterpret_cast<uint2*>(a.y16 + o) = make_uint2(lo, hi);
    }
}

struct RopeArgs {
    const float* qkv;      // [T][nqkv]: query heads, key heads, value heads
    uint16_t* q;           // [T][H][hd]
    uint16_t* kc;          // this layer's K cache [G][max_seq][hd]
    uint16_t* vc;          // this layer's V cache
    int T, H, G, hd, max_seq, pos0;
    double log_theta;
};

// one thread per (token, head slot, pair i): slot s < H is query head s,
// H <= s < H + G key head s - H, then value heads (no rotation)
__global__ __launch_bounds__(256) void rope_kernel(RopeArgs a)
{
    const int half = a.hd / 2, slots = a.H + 2 * a.G;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)a.T * slots * half) return;
    const int i = (int)(idx % half);
    const int s = (int)((idx / half) % slots);
    const int t = (int)(idx / ((int64_t)half * slots));
    const int nqkv = slots * a.hd;
    const float* src = a.qkv + (int64_t)t * nqkv + (int64_t)s * a.hd;
    const int pos = a.pos0 + t;
    const float x0 = src[i], x1 = src[i + half];
    uint16_t* dst;
    if (s >= a.H + a.G) {
        dst = a.vc + ((int64_t)(s - a.H - a.G) * a.max_seq + pos) * a.hd;
        dst[i] = moe::f32_to_bf16(x0);
        dst[i + half] = moe::f32_to_bf16(x1);
        return;
    }
    // angle pos * theta^(-2i/hd), in fp64
    const double ang = (double)pos * exp(-(2.0 * i / a.hd) * a.log_theta);
    double sn, cs;
    sincos(ang, &sn, &cs);
    const float c = (float)cs, sf = (float)sn;
    const float r0 = x0 * c - x1 * sf;
    const float r1 = x1 * c + x0 * sf;
    if (s < a.H)
        dst = a.q + ((int64_t)t * a.H + s) * a.hd;
    else
        dst = a.kc + ((int64_t)(s - a.H) * a.max_seq + pos) * a.hd;
    dst[i] = moe::f32_to_bf16(r0);
    dst[i + half] = moe::f32_to_bf16(r1);
}

struct ScoreArgs {
    const uint16_t* q;     // [T][H][hd] bf16
    const uint16_t* kc;    // [G][max_seq][hd]
    const uint16_t* vc;
    float* part;           // [T][H][n_chunks][hd + kPartPad]: sum of p v, then m, l
    int T, H, G, max_seq, pos0, n_chunks;
    float scale;           // 1 / sqrt(hd)
};

// Workgroup (key/value head g, chunk c): thread p owns position
// c * 256 + p.  The query rows are every (token t, query head j of g); row
// r's positions end at pos0 + t (causal).  Per batch of 16 rows: scores in
// fp32 (q . k in index order, times the scale), the chunk's maximum and the
// sum of exp(s - max) per row (fixed-order reductions), P in LDS, then
// thread (row, 8 or 4 dims) sums P v over the chunk's positions in order.
template <int HD>
__global__ __launch_bounds__(kChunk) void score_kernel(ScoreArgs a)
{
    __shared__ uint16_t qs[kMaxRows][HD];                 // query rows (bf16)
    __shared__ uint16_t vs[kChunk][HD];                   // the chunk's values
    __shared__ float ps[kRowBatch][kChunk];               // exp(s - max) of a batch
    __shared__ float red[4][kRowBatch];
    const int g = blockIdx.x, c = blockIdx.y;
    const int group = a.H / a.G;
    const int R = a.T * group;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int pos = c * kChunk + tid;
    const int n_pos = a.pos0 + a.T;
    // query rows r = t * group + jj -> head j = g * group + jj
    for (int e = tid; e < R * HD / 8; e += kChunk) {
        const int r = e / (HD / 8), k8 = e % (HD / 8);
        const int t = r / group, j = g * group + r % group;
        *reinterpret_cast<u32x4_t*>(&qs[r][k8 * 8]) =
            ld16(a.q + ((int64_t)t * a.H + j) * HD + k8 * 8);
    }
    u32x4_t kreg[HD / 8];
    const bool live = pos < n_pos;
    const uint16_t* kp = a.kc + ((int64_t)g * a.max_seq + (live ? pos : 0)) * HD;
    const uint16_t* vp = a.vc + ((int64_t)g * a.max_seq + (live ? pos : 0)) * HD;
#pragma unroll
    for (int k8 = 0; k8 < HD / 8; ++k8) {
        const u32x4_t zero = {0u, 0u, 0u, 0u};
        kreg[k8] = live ? ld16(kp + k8 * 8) : zero;
        *reinterpret_cast<u32x4_t*>(&vs[tid][k8 * 8]) = live ? ld16(vp + k8 * 8) : zero;
    }
    __syncthreads();
    for (int b0 = 0; b0 < R; b0 += kRowBatch) {
        float s[kRowBatch];
#pragma unroll
        for (int rr = 0; rr < kRowBatch; ++rr) {
            const int r = b0 + rr;
            float acc = 0.f;
            if (r < R) {
#pragma unroll
                for (int k8 = 0; k8 < HD / 8; ++k8) {
                    const u32x4_t qv = *reinterpret_cast<const u32x4_t*>(&qs[r][k8 * 8]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        acc = fmaf(__uint_as_float(qv[e] << 16), __uint_as_float(kreg[k8][e] << 16), acc);
                        acc = fmaf(__uint_as_float(qv[e] & 0xFFFF0000u),
                                   __uint_as_float(kreg[k8][e] & 0xFFFF0000u), acc);
                    }
                }
            }
            const bool ok = r < R && pos <= a.pos0 + r / group;
            s[rr] = ok ? acc * a.scale : -INFINITY;
        }
        // per row: the chunk maximum over the 256 positions
        float m[kRowBatch];
#pragma unroll
        for (int rr = 0; rr < kRowBatch; ++rr) {
            float v = s[rr];
            for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
            if (lane == 0) red[w][rr] = v;
        }
        __syncthreads();
#pragma unroll
        for (int rr = 0; rr < kRowBatch; ++rr)
            m[rr] = fmaxf(fmaxf(red[0][rr], red[1][rr]), fmaxf(red[2][rr], red[3][rr]));
        __syncthreads();
#pragma unroll
        for (int rr = 0; rr < kRowBatch; ++rr) {
            const float p = s[rr] == -INFINITY ? 0.f : expf(s[rr] - m[rr]);
            ps[rr][tid] = p;
            float v = p;
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
            if (lane == 0) red[w][rr] = v;
        }
        __syncthreads();
        // thread (row rr, dims dg * D .. +D-1), D = HD / 16
        constexpr int D = HD / 16;
        const int rr = tid / 16, dg = tid % 16;
        const int r = b0 + rr;
        if (r < R) {
            float acc[D];
#pragma unroll
            for (int e = 0; e < D; ++e) acc[e] = 0.f;
            const int last = min(kChunk, n_pos - c * kChunk);
            for (int p = 0; p < last; ++p) {
                const float pv = ps[rr][p];
#pragma unroll
                for (int e = 0; e < D; ++e)
                    acc[e] = fmaf(pv, __uint_as_float((uint32_t)vs[p][dg * D + e] << 16), acc[e]);
            }
            const int t = r / group, j = g * group + r % group;
            float* out = a.part + (((int64_t)t * a.H + j) * a.n_chunks + c) * (HD + kPartPad);
#pragma unroll
            for (int e = 0; e < D; ++e) out[dg * D + e] = acc[e];
            if (dg == 0) {
                out[HD] = m[rr];
                out[HD + 1] = ((red[0][rr] + red[1][rr]) + red[2][rr]) + red[3][rr];
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
    const float* base = a.part + (int64_t)th * a.n_chunks * (a.hd + kPartPad);
    float M = -INFINITY;
    for (int c = 0; c < used; ++c) M = fmaxf(M, base[(int64_t)c * (a.hd + kPartPad) + a.hd]);
    float L = 0.f, acc = 0.f;
    for (int c = 0; c < used; ++c) {
        const float* pc = base + (int64_t)c * (a.hd + kPartPad);
        const float f = expf(pc[a.hd] - M);
        L = fmaf(pc[a.hd + 1], f, L);
        acc = fmaf(pc[i], f, acc);
    }
    a.out[(int64_t)th * a.hd + i] = moe::f32_to_bf16(acc / L);
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

hipError_t attn_launch_gemv(int out_mode, const void* w, const uint16_t* x, int T, int K, int N,
                            float* y32, const uint16_t* res, uint16_t* y16, hipStream_t s)
{
    attn::GemvArgs a{static_cast<const uint8_t*>(w), x, y32, res, y16, K, N, T};
    if (out_mode)
        hipLaunchKernelGGL(attn::gemv_kernel<attn::kOut>, dim3(N / moe::kTileRows),
                           dim3(64 * attn::kSplit), 0, s, a);
    else
        hipLaunchKernelGGL(attn::gemv_kernel<attn::kQkv>, dim3(N / moe::kTileRows),
                           dim3(64 * attn::kSplit), 0, s, a);
    return hipGetLastError();
}

hipError_t attn_launch_rope(const float* qkv, uint16_t* q, uint16_t* kc, uint16_t* vc, int T,
                            int H, int G, int hd, int max_seq, int pos0, double theta,
                            hipStream_t s)
{
    attn::RopeArgs a{qkv, q, kc, vc, T, H, G, hd, max_seq, pos0, log(theta)};
    const int64_t n = (int64_t)T * (H + 2 * G) * (hd / 2);
    hipLaunchKernelGGL(attn::rope_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
    return hipGetLastError();
}

int attn_chunks(int n_pos) { return (n_pos + attn::kChunk - 1) / attn::kChunk; }
int attn_part_stride(int hd) { return hd + attn::kPartPad; }

hipError_t attn_launch_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                                 float* part, uint16_t* out, int T, int H, int G, int hd,
                                 int max_seq, int pos0, int n_chunks_alloc, hipStream_t s)
{
    const int n_chunks = attn_chunks(pos0 + T);
    attn::ScoreArgs a{q, kc, vc, part, T, H, G, max_seq, pos0, n_chunks_alloc,
                      (float)(1.0 / sqrt((double)hd))};
    if (hd == 128)
        hipLaunchKernelGGL(attn::score_kernel<128>, dim3(G, n_chunks), dim3(attn::kChunk), 0, s, a);
    else
        hipLaunchKernelGGL(attn::score_kernel<64>, dim3(G, n_chunks), dim3(attn::kChunk), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    attn::CombineArgs c{part, out, H, hd, pos0, n_chunks_alloc};
    hipLaunchKernelGGL(attn::combine_kernel, dim3(T * H), dim3(128), 0, s, c);
    return hipGetLastError();
}

}  // extern "C"
