// moe_route.hip -- the router (paper Sec. 3.1: its output decides which
// experts receive a token), top-k selection (Sec. 2.1: 4 of 16), the gate
// weights, and the token -> expert permutation.
//
// Logits.  The product of a bf16 activation and an fp32 router weight is
// exact in fp64, so the kernels accumulate in fp64 and round once to fp32:
// the logit equals the fp32 rounding of the exact dot product except when
// that sum lies within a few fp64 ulps of an fp32 rounding boundary.  The
// router weight is held transposed in the arena (wrT [E][d], d contiguous) so
// that every load is 16 bytes.
//
// Kernels
//   route_small_kernel  (T <= kSmallT): one 1024-thread workgroup computes the
//       logits (thread = expert x d-slice, fixed-order LDS reduction), then
//       selects, weighs and permutes -- a single launch for a decode step.
//   router_logits_kernel (larger T): 4 tokens per 256-thread workgroup, each
//       (token, expert) dot product split over four threads and summed in
//       fixed order through LDS.
//   route_decode_kernel (T <= 16, E <= 16, T*k <= 64): the logits spread over
//       d/512 workgroups, the last one to finish selects and permutes.
//   route_kernel: selection, weights and permutation from fp32 logits.
//
// Selection: the k largest logits, ties to the lower expert id, slots ordered
// by (logit desc, id asc); weights = softmax over the selected logits (fp32).
// Permutation: block-wide prefix sums per local expert over pairs in (token,
// slot) order, which gives rows grouped by expert, then token -- no atomics,
// so the order is deterministic.
#include <algorithm>

#include "moe_common.h"

namespace moe {

constexpr int kRouteThreads = 1024;
constexpr int kRouteWaves = kRouteThreads / kWave;
constexpr int kSmallPartials = 4096;   // doubles of LDS for the slice partials

struct RouteArgs {
    const uint16_t* x;        // [T, d]          (route_small_kernel)
    const float* wrT;         // [E, d]          (route_small_kernel)
    const float* logits_in;   // [T, E] or null  (route_kernel: read from here if set)
    const float* bias;        // [E] or null     (route_small_kernel)
    int T, d, E, k;
    int e_begin, n_local;
    int tile_rows;            // token rows per GEMM tile
    RouteView rv;
};

// Selection and weights for token t from logits l[0..E) (any address space).
// The logits, the chosen ids and their exponentials stay in registers
// (kMaxE and kMaxK bound the static arrays; E <= 64 always).
constexpr int kMaxK = 8;

template <int kMaxE>
__device__ inline void select_token(const float* l, int t, int E, int k, const RouteView& rv)
{
    float lv[kMaxE];
#pragma unroll
    for (int e = 0; e < kMaxE; ++e) lv[e] = e < E ? l[e] : 0.f;
    uint64_t taken = 0;
    int ids[kMaxK];
    float ps[kMaxK];
    float lmax = 0.f, z = 0.f;
    for (int j = 0; j < k; ++j) {
        int best = -1;
        float bv = 0.f;
#pragma unroll
        for (int e = 0; e < kMaxE; ++e) {
            const bool ok = e < E && !((taken >> e) & 1ull);
            if (ok && (best < 0 || lv[e] > bv)) { best = e; bv = lv[e]; }
        }
        taken |= 1ull << best;
        if (j == 0) lmax = bv;
        const float p = expf(bv - lmax);
        z += p;
        rv.topk_idx[(int64_t)t * k + j] = best;
#pragma unroll
        for (int q = 0; q < kMaxK; ++q)
            if (q == j) { ids[q] = best; ps[q] = p; }
        if (j >= kMaxK) rv.topk_w[(int64_t)t * k + j] = p;   // normalised below
    }
    const float inv = 1.0f / z;
#pragma unroll
    for (int q = 0; q < kMaxK; ++q)
        if (q < k) rv.topk_w[(int64_t)t * k + q] = ps[q] * inv;
    for (int j = kMaxK; j < k; ++j) {
        float* pw = rv.topk_w + (int64_t)t * k + j;
        *pw = *pw * inv;
    }
    (void)ids;
}

__device__ inline void select_token_any(const float* l, int t, int E, int k, const RouteView& rv)
{
    if (E <= 16) select_token<16>(l, t, E, k, rv);
    else select_token<64>(l, t, E, k, rv);
}

// Expert-grouped permutation of the T*k pairs (whole workgroup); needs the
// workgroup's topk_idx writes to be visible (caller syncs).  Each thread owns
// a contiguous chunk of pairs; per group of 16 experts, every thread counts
// its pairs per expert, a wave-level inclusive scan and one LDS pass over the
// wave totals give each thread its first row per expert, and the thread then
// writes its rows -- three barriers per expert group.
constexpr int kPermExperts = 16;
constexpr int kPermMaxChunk = 8;

__device__ void build_permutation(const RouteArgs& a, int (*lds_tot)[kPermExperts],
                                  int* lds_counts)
{
    const int T = a.T, E = a.E, k = a.k;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const RouteView& rv = a.rv;
    const int P = T * k;
    const int chunk = (P + kRouteThreads - 1) / kRouteThreads;
    const int p0 = min(P, tid * chunk);
    const int p1 = min(P, p0 + chunk);
    const int lo = a.e_begin, hi = a.e_begin + a.n_local;
    // the chunk's expert ids, held in registers when the chunk is short
    int ids[kPermMaxChunk];
    const bool in_regs = chunk <= kPermMaxChunk;
#pragma unroll
    for (int q = 0; q < kPermMaxChunk; ++q)
        ids[q] = (in_regs && p0 + q < p1) ? rv.topk_idx[p0 + q] : -1;
    auto id_at = [&](int p) {
        if (in_regs) {
            int v = -1;
#pragma unroll
            for (int q = 0; q < kPermMaxChunk; ++q)
                if (p - p0 == q) v = ids[q];
            return v;
        }
        return rv.topk_idx[p];
    };
    for (int p = p0; p < p1; ++p) {
        const int e = id_at(p);
        if (e < lo || e >= hi) rv.pair_row[p] = -1;
    }
    int running = 0;   // rows of all earlier experts
    for (int e0 = 0; e0 < E; e0 += kPermExperts) {
        int cnt[kPermExperts];
#pragma unroll
        for (int j = 0; j < kPermExperts; ++j) cnt[j] = 0;
        for (int p = p0; p < p1; ++p) {
            const int e = id_at(p);
#pragma unroll
            for (int j = 0; j < kPermExperts; ++j) cnt[j] += (e == e0 + j) ? 1 : 0;
        }
        // wave-level inclusive scans of the 16 counters
        int inc[kPermExperts];
#pragma unroll
        for (int j = 0; j < kPermExperts; ++j) {
            int v = cnt[j];
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int o = __shfl_up(v, off, 64);
                if (lane >= off) v += o;
            }
            inc[j] = v;
        }
        if (lane == 63) {
#pragma unroll
            for (int j = 0; j < kPermExperts; ++j) lds_tot[wid][j] = inc[j];
        }
        __syncthreads();
        int base[kPermExperts];
        int run = running;
#pragma unroll
        for (int j = 0; j < kPermExperts; ++j) {
            const int e = e0 + j;
            int before = 0, tot = 0;
            for (int w = 0; w < kRouteWaves; ++w) {
                const int c = lds_tot[w][j];
                before += (w < wid) ? c : 0;
                tot += c;
            }
            const bool local = e < E && e >= lo && e < hi;
            if (!local) tot = 0;
            base[j] = run + before + inc[j] - cnt[j];
            if (tid == 0 && e < E) {
                rv.counts[e] = tot;
                rv.offsets[e] = run;
                lds_counts[e] = tot;
            }
            run += tot;
        }
        for (int p = p0; p < p1; ++p) {
            const int e = id_at(p);
            if (e >= e0 && e < e0 + kPermExperts && e >= lo && e < hi) {
                int r = 0;
#pragma unroll
                for (int j = 0; j < kPermExperts; ++j)
                    if (e == e0 + j) r = base[j]++;
                rv.pair_row[p] = r;
                rv.row_token[r] = p / k;
            }
        }
        running = run;
        __syncthreads();
    }
    if (tid == 0) {
        rv.offsets[E] = running;
        int na = 0, nt = 0, row = 0;
        for (int e = 0; e < E; ++e) {
            const int c = lds_counts[e];
            if (c > 0) {
                rv.active[1 + na++] = e;
                for (int r = 0; r < c; r += a.tile_rows) {
                    rv.tiles[2 * nt] = e;
                    rv.tiles[2 * nt + 1] = row + r;
                    ++nt;
                }
            }
            row += c;
        }
        rv.active[0] = na;
        *rv.n_tiles = nt;
    }
}

__device__ inline void fma8(double& acc, const u32x4_t xv, const float4 w0, const float4 w1)
{
    acc = fma((double)__uint_as_float(xv[0] << 16), (double)w0.x, acc);
    acc = fma((double)__uint_as_float(xv[0] & 0xFFFF0000u), (double)w0.y, acc);
    acc = fma((double)__uint_as_float(xv[1] << 16), (double)w0.z, acc);
    acc = fma((double)__uint_as_float(xv[1] & 0xFFFF0000u), (double)w0.w, acc);
    acc = fma((double)__uint_as_float(xv[2] << 16), (double)w1.x, acc);
    acc = fma((double)__uint_as_float(xv[2] & 0xFFFF0000u), (double)w1.y, acc);
    acc = fma((double)__uint_as_float(xv[3] << 16), (double)w1.z, acc);
    acc = fma((double)__uint_as_float(xv[3] & 0xFFFF0000u), (double)w1.w, acc);
}

constexpr int kSmallT = 16;

__global__ __launch_bounds__(kRouteThreads) void route_small_kernel(RouteArgs a)
{
    __shared__ double part[kSmallPartials];
    __shared__ float lg[kSmallT * 64];
    __shared__ int lds_tot[kRouteWaves][kPermExperts];
    __shared__ int lds_counts[64];
    const int T = a.T, E = a.E, d = a.d;
    const int tid = threadIdx.x;

    // slices: S slices of the d axis per expert, S*T*E partials fit in LDS
    int S = kRouteThreads / E;
    while (S > 1 && S * T * E > kSmallPartials) S >>= 1;
    const int groups = d / 8;                         // 8-element groups
    const int per = (groups + S - 1) / S;             // groups per slice
    if (tid < E * S) {
        const int e = tid % E;
        const int s = tid / E;
        const int g0 = s * per;
        const int g1 = min(groups, g0 + per);
        double acc[kSmallT];
#pragma unroll
        for (int t = 0; t < kSmallT; ++t) acc[t] = 0.0;
        const float* wrow = a.wrT + (int64_t)e * d;
#pragma unroll 6
        for (int g = g0; g < g1; ++g) {
            const float4 w0 = *reinterpret_cast<const float4*>(wrow + g * 8);
            const float4 w1 = *reinterpret_cast<const float4*>(wrow + g * 8 + 4);
#pragma unroll
            for (int t = 0; t < kSmallT; ++t) {
                if (t < T) {
                    const u32x4_t xv = *reinterpret_cast<const u32x4_t*>(a.x + (int64_t)t * d + g * 8);
                    fma8(acc[t], xv, w0, w1);
                }
            }
        }
#pragma unroll
        for (int t = 0; t < kSmallT; ++t)
            if (t < T) part[(s * T + t) * E + e] = acc[t];
    }
    __syncthreads();
    if (tid < T * E) {
        const int t = tid / E, e = tid % E;
        double sum = 0.0;
        for (int s = 0; s < S; ++s) sum += part[(s * T + t) * E + e];
        float v = (float)sum;
        if (a.bias) v = __fadd_rn(v, a.bias[e]);
        lg[t * 64 + e] = v;
        a.rv.logits[(int64_t)t * E + e] = v;
    }
    __syncthreads();
    if (tid < T) select_token_any(&lg[tid * 64], tid, E, a.k, a.rv);
    __syncthreads();
    build_permutation(a, lds_tot, lds_counts);
}

// Decode routing (T <= 16, E <= 16, T*k <= 64): the logits are spread over
// n_wg workgroups, each owning d/n_wg of the reduction axis (one 8-wide group
// per thread, thread = (expert tid%16, group tid/16)).  Per workgroup the
// partials are reduced in fixed order (lane butterfly, then over the 16 waves
// through LDS) and written to the workspace; the workgroup that takes the last
// ticket of a device-scope counter sums the n_wg partials in workgroup order,
// selects, weighs and permutes, and rewinds the counter for the next call.
constexpr int kDecE = 16;
constexpr int kDecPairs = 64;

struct DecodeRouteArgs {
    const uint16_t* x;
    const float* wrT;
    const float* bias;
    double* partial;          // [n_wg][kSmallT][kDecE]
    unsigned int* counter;    // one device-scope ticket counter (0 between calls)
    int T, d, E, k, e_begin, n_local, tile_rows, n_wg;
    RouteView rv;
};

__global__ __launch_bounds__(kRouteThreads) void route_decode_kernel(DecodeRouteArgs a)
{
    __shared__ double wsum[kRouteWaves][kSmallT][kDecE];
    __shared__ float lg[kSmallT][kDecE];
    __shared__ int s_ids[kDecPairs];
    __shared__ int s_cnt[kDecE];
    __shared__ int s_off[kDecE + 1];
    __shared__ int s_last;
    const int T = a.T, E = a.E, d = a.d, k = a.k;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int e = tid & 15;
    const int g = blockIdx.x * (kRouteThreads / kDecE) + (tid >> 4);
    double acc[kSmallT];
#pragma unroll
    for (int t = 0; t < kSmallT; ++t) acc[t] = 0.0;
    if (e < E && g < d / 8) {
        const float4 w0 = *reinterpret_cast<const float4*>(a.wrT + (int64_t)e * d + g * 8);
        const float4 w1 = *reinterpret_cast<const float4*>(a.wrT + (int64_t)e * d + g * 8 + 4);
#pragma unroll
        for (int t = 0; t < kSmallT; ++t)
            if (t < T)
                fma8(acc[t], *reinterpret_cast<const u32x4_t*>(a.x + (int64_t)t * d + g * 8), w0, w1);
    }
    // lanes l, l^16, l^32, l^48 hold the same expert: fixed-order butterfly
#pragma unroll
    for (int t = 0; t < kSmallT; ++t) {
        if (t < T) {
            double v = acc[t];
            v += __shfl_xor(v, 16, 64);
            v += __shfl_xor(v, 32, 64);
            if (lane < kDecE) wsum[wid][t][lane] = v;
        }
    }
    __syncthreads();
    if (tid < T * kDecE) {
        const int t = tid / kDecE, ee = tid % kDecE;
        double v = 0.0;
        for (int w = 0; w < kRouteWaves; ++w) v += wsum[w][t][ee];
        a.partial[((int64_t)blockIdx.x * kSmallT + t) * kDecE + ee] = v;
    }
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(a.counter, 1u) == (unsigned)(a.n_wg - 1)) ? 1 : 0;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    if (tid < T * kDecE) {
        const int t = tid / kDecE, ee = tid % kDecE;
        if (ee < E) {
            double v = 0.0;
            for (int w = 0; w < a.n_wg; ++w)
                v += __builtin_nontemporal_load(&a.partial[((int64_t)w * kSmallT + t) * kDecE + ee]);
            float l = (float)v;
            if (a.bias) l = __fadd_rn(l, a.bias[ee]);
            lg[t][ee] = l;
            a.rv.logits[(int64_t)t * E + ee] = l;
        }
    }
    if (tid == 0) *a.counter = 0u;
    __syncthreads();
    // selection (one thread per token); ids also kept in LDS
    if (tid < T) {
        select_token<kDecE>(&lg[tid][0], tid, E, k, a.rv);
        for (int j = 0; j < k; ++j) s_ids[tid * k + j] = a.rv.topk_idx[(int64_t)tid * k + j];
    }
    __syncthreads();
    const int P = T * k;
    const int lo = a.e_begin, hi = a.e_begin + a.n_local;
    if (tid < E) {
        int c = 0;
        if (tid >= lo && tid < hi)
            for (int p = 0; p < P; ++p) c += (s_ids[p] == tid);
        s_cnt[tid] = c;
    }
    __syncthreads();
    if (tid == 0) {
        int run = 0, na = 0, nt = 0;
        for (int ee = 0; ee < E; ++ee) {
            const int c = s_cnt[ee];
            s_off[ee] = run;
            a.rv.counts[ee] = c;
            a.rv.offsets[ee] = run;
            if (c > 0) {
                a.rv.active[1 + na++] = ee;
                for (int r = 0; r < c; r += a.tile_rows) {
                    a.rv.tiles[2 * nt] = ee;
                    a.rv.tiles[2 * nt + 1] = run + r;
                    ++nt;
                }
            }
            run += c;
        }
        s_off[E] = run;
        a.rv.offsets[E] = run;
        a.rv.active[0] = na;
        *a.rv.n_tiles = nt;
    }
    __syncthreads();
    if (tid < P) {
        const int ee = s_ids[tid];
        if (ee >= lo && ee < hi) {
            int rank = 0;
            for (int p = 0; p < tid; ++p) rank += (s_ids[p] == ee);
            const int r = s_off[ee] + rank;
            a.rv.pair_row[tid] = r;
            a.rv.row_token[r] = tid / k;
        } else {
            a.rv.pair_row[tid] = -1;
        }
    }
}

__global__ void zero_u32_kernel(unsigned int* p) { *p = 0u; }

// logits for 4 tokens per workgroup: thread = (d-split tid/64, token
// (tid/16)%4, expert slot tid%16) over experts slot, slot+16, ...; each thread
// streams a quarter of the token row and of the expert row in 16-byte vectors
// with two interleaved accumulators, and the four quarter sums are added in
// split order through LDS.
constexpr int kLogitTok = 4;
constexpr int kLogitSplit = 4;

__global__ __launch_bounds__(256) void router_logits_kernel(const uint16_t* __restrict__ x,
                                                            const float* __restrict__ wrT,
                                                            const float* __restrict__ bias, int T,
                                                            int d, int E,
                                                            float* __restrict__ logits)
{
    __shared__ double part[kLogitSplit][kLogitTok][64];
    const int tid = threadIdx.x;
    const int sp = tid >> 6;
    const int tl = (tid >> 4) & 3;
    const int es = tid & 15;
    const int t = blockIdx.x * kLogitTok + tl;
    const int q = d / kLogitSplit;            // d is a multiple of 256
    if (t < T) {
        const uint16_t* xr = x + (int64_t)t * d + sp * q;
        for (int e = es; e < E; e += 16) {
            const float* wr = wrT + (int64_t)e * d + sp * q;
            double a0 = 0.0, a1 = 0.0;
#pragma unroll 8
            for (int g = 0; g < q; g += 16) {
                const u32x4_t x0 = *reinterpret_cast<const u32x4_t*>(xr + g);
                const u32x4_t x1 = *reinterpret_cast<const u32x4_t*>(xr + g + 8);
                const float4 w0 = *reinterpret_cast<const float4*>(wr + g);
                const float4 w1 = *reinterpret_cast<const float4*>(wr + g + 4);
                const float4 w2 = *reinterpret_cast<const float4*>(wr + g + 8);
                const float4 w3 = *reinterpret_cast<const float4*>(wr + g + 12);
                fma8(a0, x0, w0, w1);
                fma8(a1, x1, w2, w3);
            }
            part[sp][tl][e] = a0 + a1;
        }
    }
    __syncthreads();
    if (sp == 0 && t < T) {
        for (int e = es; e < E; e += 16) {
            double s = part[0][tl][e];
            for (int k = 1; k < kLogitSplit; ++k) s += part[k][tl][e];
            float v = (float)s;
            if (bias) v = __fadd_rn(v, bias[e]);
            logits[(int64_t)t * E + e] = v;
        }
    }
}

__global__ __launch_bounds__(kRouteThreads) void route_kernel(RouteArgs a)
{
    __shared__ int lds_tot[kRouteWaves][kPermExperts];
    __shared__ int lds_counts[64];
    const float* src = a.logits_in ? a.logits_in : a.rv.logits;
    for (int t = threadIdx.x; t < a.T; t += kRouteThreads) {
        if (a.logits_in)
            for (int e = 0; e < a.E; ++e)
                a.rv.logits[(int64_t)t * a.E + e] = src[(int64_t)t * a.E + e];
        select_token_any(src + (int64_t)t * a.E, t, a.E, a.k, a.rv);
    }
    __syncthreads();
    build_permutation(a, lds_tot, lds_counts);
}

// wrT[e][i] = wr[i][e]
__global__ __launch_bounds__(256) void transpose_router_kernel(const float* __restrict__ wr, int d,
                                                               int E, float* __restrict__ wrT)
{
    const int64_t n = (int64_t)d * E;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < n;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = o / d, i = o % d;
        wrT[o] = wr[i * E + e];
    }
}

}  // namespace moe

extern "C" int moe_route_small_max_tokens() { return moe::kSmallT; }

extern "C" hipError_t moe_launch_route_small(const uint16_t* x, const float* wrT,
                                             const float* bias, int T, int d, int E, int k,
                                             int e_begin, int n_local, int tile_rows,
                                             const moe::RouteView* rv, hipStream_t s)
{
    moe::RouteArgs a{};
    a.x = x; a.wrT = wrT; a.logits_in = nullptr; a.bias = bias;
    a.T = T; a.d = d; a.E = E; a.k = k;
    a.e_begin = e_begin; a.n_local = n_local; a.tile_rows = tile_rows;
    a.rv = *rv;
    hipLaunchKernelGGL(moe::route_small_kernel, dim3(1), dim3(moe::kRouteThreads), 0, s, a);
    return hipGetLastError();
}

extern "C" int moe_route_decode_ok(int T, int E, int k)
{
    return T >= 1 && T <= moe::kSmallT && E <= moe::kDecE && T * k <= moe::kDecPairs;
}

extern "C" int moe_route_decode_wgs(int d) { return (d / 8 + 63) / 64; }

extern "C" hipError_t moe_launch_zero_counter(unsigned int* counter, hipStream_t s)
{
    hipLaunchKernelGGL(moe::zero_u32_kernel, dim3(1), dim3(1), 0, s, counter);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_route_decode(const uint16_t* x, const float* wrT,
                                              const float* bias, double* partial,
                                              unsigned int* counter, int T, int d, int E, int k,
                                              int e_begin, int n_local, int tile_rows,
                                              const moe::RouteView* rv, hipStream_t s)
{
    moe::DecodeRouteArgs a{};
    a.x = x; a.wrT = wrT; a.bias = bias; a.partial = partial; a.counter = counter;
    a.T = T; a.d = d; a.E = E; a.k = k;
    a.e_begin = e_begin; a.n_local = n_local; a.tile_rows = tile_rows;
    a.n_wg = moe_route_decode_wgs(d);
    a.rv = *rv;
    hipLaunchKernelGGL(moe::route_decode_kernel, dim3(a.n_wg), dim3(moe::kRouteThreads), 0, s, a);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_router_logits(const uint16_t* x, const float* wrT,
                                               const float* bias, int T, int d, int E,
                                               float* logits, hipStream_t s)
{
    const int grid = (T + moe::kLogitTok - 1) / moe::kLogitTok;
    hipLaunchKernelGGL(moe::router_logits_kernel, dim3(grid), dim3(256), 0, s, x, wrT, bias, T, d,
                       E, logits);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_route(const float* logits_in, int T, int E, int k, int e_begin,
                                       int n_local, int tile_rows, const moe::RouteView* rv,
                                       hipStream_t s)
{
    moe::RouteArgs a{};
    a.logits_in = logits_in;
    a.T = T; a.E = E; a.k = k;
    a.e_begin = e_begin; a.n_local = n_local; a.tile_rows = tile_rows;
    a.rv = *rv;
    hipLaunchKernelGGL(moe::route_kernel, dim3(1), dim3(moe::kRouteThreads), 0, s, a);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_transpose_router(const float* wr, int d, int E, float* wrT,
                                                  hipStream_t s)
{
    const int64_t n = (int64_t)d * E;
    int grid = (int)std::min<int64_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(moe::transpose_router_kernel, dim3(grid), dim3(256), 0, s, wr, d, E, wrT);
    return hipGetLastError();
}
