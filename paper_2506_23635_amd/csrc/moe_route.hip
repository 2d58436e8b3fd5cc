// moe_route.hip -- the router (paper Sec. 3.1: its output decides which
// experts receive a token), top-k selection (Sec. 2.1: 4 of 16), the gate
// weights, and the token -> expert permutation.
//
// router_partial_kernel: logits as fp64 partial dot products over d-slices.
//   The product of a bf16 and an fp32 is exact in fp64, so the fp64 sum is
//   the exact dot product up to fp64 rounding, and one final rounding to
//   fp32 gives the logit; bit-identical to rounding the exact sum except in
//   cases within a few fp64 ulps of an fp32 rounding boundary.
// route_kernel: one 1024-thread workgroup.  Sums the slices in fixed order,
//   rounds to fp32, adds the bias in fp32, selects the top-k (logit desc, id
//   asc), computes the softmax of the selected logits in fp32, then builds the
//   stable expert-grouped permutation with block-wide prefix sums (no atomics,
//   so the row order is deterministic) and the per-expert token tiles that the
//   grouped GEMM walks.
#include "moe_common.h"

namespace moe {

// thread <-> (slice s, token t, expert e); partial[s][t][e] = sum over the
// slice of x[t,i] * wr[i,e] in fp64.
__global__ __launch_bounds__(256) void router_partial_kernel(const uint16_t* __restrict__ x,
                                                             const float* __restrict__ wr, int T,
                                                             int d, int E, int n_slices,
                                                             int slice_len,
                                                             double* __restrict__ partial)
{
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)n_slices * T * E;
    if (gid >= total) return;
    const int e = (int)(gid % E);
    const int t = (int)((gid / E) % T);
    const int s = (int)(gid / ((int64_t)E * T));
    const int i0 = s * slice_len;
    const int i1 = min(d, i0 + slice_len);
    const uint16_t* xr = x + (int64_t)t * d;
    double acc = 0.0;
    for (int i = i0; i < i1; ++i)
        acc = fma((double)bf16_to_f32(xr[i]), (double)wr[(int64_t)i * E + e], acc);
    partial[gid] = acc;
}

constexpr int kRouteThreads = 1024;
constexpr int kRouteWaves = kRouteThreads / kWave;

// Block-wide exclusive scan of one int per thread; returns the exclusive
// prefix, writes the block total to *total.  Uses the wave prefix via shuffles.
__device__ inline int block_exclusive_scan(int v, int* lds_wave, int* total)
{
    const int lane = threadIdx.x & 63;
    const int wid = threadIdx.x >> 6;
    int inc = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int o = __shfl_up(inc, off, 64);
        if (lane >= off) inc += o;
    }
    if (lane == 63) lds_wave[wid] = inc;
    __syncthreads();
    int base = 0, tot = 0;
    for (int w = 0; w < kRouteWaves; ++w) {
        int c = lds_wave[w];
        if (w < wid) base += c;
        tot += c;
    }
    __syncthreads();
    *total = tot;
    return base + inc - v;
}

struct RouteArgs {
    const double* partial;   // [n_slices][T][E] or null when logits_in is given
    const float* logits_in;  // [T][E] or null
    const float* bias;       // [E] or null
    int n_slices;
    int T, E, k;
    int e_begin, n_local;
    int tile_rows;           // token rows per GEMM tile
    RouteView rv;
};

__global__ __launch_bounds__(kRouteThreads) void route_kernel(RouteArgs a)
{
    __shared__ int lds_wave[kRouteWaves];
    __shared__ int lds_counts[64];
    const int T = a.T, E = a.E, k = a.k;
    const int tid = threadIdx.x;

    // 1) logits, selection, weights: one token per thread
    for (int t = tid; t < T; t += kRouteThreads) {
        float l[64];
        for (int e = 0; e < E; ++e) {
            float v;
            if (a.logits_in) {
                v = a.logits_in[(int64_t)t * E + e];
            } else {
                double s = 0.0;
                for (int sl = 0; sl < a.n_slices; ++sl)
                    s += a.partial[((int64_t)sl * T + t) * E + e];
                v = (float)s;
                if (a.bias) v = __fadd_rn(v, a.bias[e]);
            }
            l[e] = v;
            a.rv.logits[(int64_t)t * E + e] = v;
        }
        uint64_t taken = 0;
        float lmax = 0.f, z = 0.f;
        float sel[64];
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                if ((taken >> e) & 1ull) continue;
                if (best < 0 || l[e] > l[best]) best = e;
            }
            taken |= 1ull << best;
            a.rv.topk_idx[(int64_t)t * k + j] = best;
            if (j == 0) lmax = l[best];
            sel[j] = expf(l[best] - lmax);
            z += sel[j];
        }
        for (int j = 0; j < k; ++j) a.rv.topk_w[(int64_t)t * k + j] = sel[j] / z;
    }
    __syncthreads();

    // 2) permutation: each thread owns a contiguous chunk of pairs p = t*k + j
    const int P = T * k;
    const int chunk = (P + kRouteThreads - 1) / kRouteThreads;
    const int p0 = min(P, tid * chunk);
    const int p1 = min(P, p0 + chunk);
    for (int p = p0; p < p1; ++p) {
        int e = a.rv.topk_idx[p];
        if (e < a.e_begin || e >= a.e_begin + a.n_local) a.rv.pair_row[p] = -1;
    }
    int running = 0;
    for (int e = 0; e < E; ++e) {
        if (e < a.e_begin || e >= a.e_begin + a.n_local) {
            if (tid == 0) { a.rv.counts[e] = 0; a.rv.offsets[e] = running; }
            continue;
        }
        int c = 0;
        for (int p = p0; p < p1; ++p) c += (a.rv.topk_idx[p] == e);
        int tot;
        int my = running + block_exclusive_scan(c, lds_wave, &tot);
        for (int p = p0; p < p1; ++p) {
            if (a.rv.topk_idx[p] == e) {
                a.rv.pair_row[p] = my;
                a.rv.row_token[my] = p / k;
                ++my;
            }
        }
        if (tid == 0) { a.rv.counts[e] = tot; a.rv.offsets[e] = running; }
        if (tid == 0 && e < 64) lds_counts[e] = tot;
        running += tot;
    }
    __syncthreads();
    if (tid == 0) {
        a.rv.offsets[E] = running;
        // active local experts and the GEMM token tiles, in expert order
        int na = 0, nt = 0, row = 0;
        for (int e = 0; e < E; ++e) {
            int c = (e >= a.e_begin && e < a.e_begin + a.n_local) ? lds_counts[e] : 0;
            if (c > 0) {
                a.rv.active[1 + na++] = e;
                for (int r = 0; r < c; r += a.tile_rows) {
                    a.rv.tiles[2 * nt] = e;
                    a.rv.tiles[2 * nt + 1] = row + r;
                    ++nt;
                }
            }
            row += c;
        }
        a.rv.active[0] = na;
        *a.rv.n_tiles = nt;
    }
}

}  // namespace moe

extern "C" hipError_t moe_launch_router_partial(const uint16_t* x, const float* wr, int T, int d,
                                                int E, int n_slices, double* partial,
                                                hipStream_t s)
{
    int slice_len = (d + n_slices - 1) / n_slices;
    int64_t total = (int64_t)n_slices * T * E;
    int grid = (int)((total + 255) / 256);
    hipLaunchKernelGGL(moe::router_partial_kernel, dim3(grid), dim3(256), 0, s, x, wr, T, d, E,
                       n_slices, slice_len, partial);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_route(const double* partial, const float* logits_in,
                                       const float* bias, int n_slices, int T, int E, int k,
                                       int e_begin, int n_local, int tile_rows,
                                       const moe::RouteView* rv, hipStream_t s)
{
    moe::RouteArgs a;
    a.partial = partial;
    a.logits_in = logits_in;
    a.bias = bias;
    a.n_slices = n_slices;
    a.T = T; a.E = E; a.k = k;
    a.e_begin = e_begin; a.n_local = n_local;
    a.tile_rows = tile_rows;
    a.rv = *rv;
    hipLaunchKernelGGL(moe::route_kernel, dim3(1), dim3(moe::kRouteThreads), 0, s, a);
    return hipGetLastError();
}
