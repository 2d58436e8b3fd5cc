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
//   router_select_kernel: 8 tokens per workgroup, a wave takes 4 tokens x 8
//       experts, each dot product split over the 64 lanes and summed by a
//       fixed transpose-reduce; then each token's selection.
//   route_partials_kernel + route_finish_kernel (T <= 16, E <= 16,
//       T*k <= 64): partial logits over a few workgroups, then one workgroup
//       sums them in fixed order, selects and permutes.
//   select_kernel: selection and weights from caller-supplied fp32 logits.
//   permute_kernel: the permutation and the GEMM tile list (one workgroup).
//
// Selection: the k largest logits, ties to the lower expert id, slots ordered
// by (logit desc, id asc); weights = softmax over the selected logits (fp32).
// Permutation: prefix sums per local expert over pairs in (token, slot)
// order, which gives rows grouped by expert, then token -- no atomic decides
// a row, so the order is deterministic.
#include <algorithm>

#include "moe_common.h"

namespace moe {

constexpr int kRouteThreads = 1024;
constexpr int kRouteWaves = kRouteThreads / kWave;
// Selection and weights for token t from logits l[0..E) (any address space).
// The logits, the chosen ids and their exponentials stay in registers
// (kMaxE and kMaxK bound the static arrays; E <= 64 always).
constexpr int kMaxK = 8;

template <int kMaxE>
__device__ __forceinline__ void select_token(const float* l, int E, int k, int* ids, float* w)
{
    float lv[kMaxE];
#pragma unroll
    for (int e = 0; e < kMaxE; ++e) lv[e] = e < E ? l[e] : 0.f;
    uint64_t taken = 0;
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
        ids[j] = best;
#pragma unroll
        for (int q = 0; q < kMaxK; ++q)
            if (q == j) ps[q] = p;
        if (j >= kMaxK) w[j] = p;   // normalised below
    }
    const float inv = 1.0f / z;
#pragma unroll
    for (int q = 0; q < kMaxK; ++q)
        if (q < k) w[q] = ps[q] * inv;
    for (int j = kMaxK; j < k; ++j) w[j] = w[j] * inv;
}

// selection of token t into the routing view (inlined: as a call it spills
// callee-saved registers to scratch)
__device__ __forceinline__ void select_token_any(const float* l, int t, int E, int k, const RouteView& rv)
{
    int* ids = rv.topk_idx + (int64_t)t * k;
    float* w = rv.topk_w + (int64_t)t * k;
    if (E <= 16) select_token<16>(l, E, k, ids, w);
    else select_token<64>(l, E, k, ids, w);
}

// barrier for LDS traffic only: waits for this wave's LDS operations, not for
// its outstanding global stores (which a __syncthreads() release would)
__device__ __forceinline__ void lds_barrier()
{
    constexpr int kWaitLgkm = 0xC07F;   // lgkmcnt 0; vmcnt and expcnt at their maxima
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(kWaitLgkm);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
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

// Decode routing (T <= 16, E <= 16, T*k <= 64) in two launches.
// route_partials_kernel spreads the logits over n_wg workgroups, each owning
// d/n_wg of the reduction axis (8-wide groups, thread = (expert tid%16, group
// tid/16)); per workgroup the partials are reduced in fixed order (lane
// butterfly, then over the 16 waves through LDS) and written to the
// workspace.  route_finish_kernel, one workgroup, sums the n_wg partials in
// workgroup order, selects, weighs and permutes.  The kernel boundary orders
// the two: measured, it costs less than a release fence, a device-scope
// ticket and an acquire inside one launch (~9 us of a 14 us kernel).
constexpr int kDecE = 16;
constexpr int kDecPairs = 64;
constexpr int kDecMaxWg = 16;   // partial sums read in one batch (d <= 8192)

struct DecodeRouteArgs {
    const uint16_t* x;
    const float* wrT;
    const float* bias;
    double* partial;          // [n_wg][kSmallT][kDecE]
    int T, d, E, k, e_begin, n_local, tile_rows, n_wg;
    RouteView rv;
};

__global__ __launch_bounds__(kRouteThreads) void route_partials_kernel(DecodeRouteArgs a)
{
    __shared__ double wsum[kRouteWaves][kSmallT][kDecE];
    const int T = a.T, E = a.E, d = a.d;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int e = tid & 15;
    double acc[kSmallT];
#pragma unroll
    for (int t = 0; t < kSmallT; ++t) acc[t] = 0.0;
    // 8-element groups blockIdx*64 + tid/16, then + n_wg*64, ... (one pass
    // when the grid covers d, several for a single workgroup)
    for (int g = blockIdx.x * (kRouteThreads / kDecE) + (tid >> 4); e < E && g < d / 8;
         g += a.n_wg * (kRouteThreads / kDecE)) {
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
}

// logits, selection and permutation in LDS, then every routing output
// written at the end (global stores are not waited for inside the
// workgroup).  Every step is spread over threads: one (token, expert) pair
// per thread.
__global__ __launch_bounds__(kRouteThreads) void route_finish_kernel(DecodeRouteArgs a)
{
    __shared__ float lg[kSmallT][kDecE];
    __shared__ int s_ids[kDecPairs];
    __shared__ float s_w[kDecPairs];
    __shared__ int s_rank[kSmallT][kDecE];
    __shared__ int s_cnt[kDecE];
    __shared__ int s_off[kDecE + 1];
    const int T = a.T, E = a.E, k = a.k;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    if (tid < T * kDecE) {
        const int t = tid / kDecE, ee = tid % kDecE;
        if (ee < E) {
            // the partials of all workgroups loaded at once, summed in
            // workgroup order
            double pv[kDecMaxWg];
#pragma unroll
            for (int w = 0; w < kDecMaxWg; ++w)
                pv[w] = w < a.n_wg ? __builtin_nontemporal_load(
                                         &a.partial[((int64_t)w * kSmallT + t) * kDecE + ee])
                                   : 0.0;
            double v = 0.0;
#pragma unroll
            for (int w = 0; w < kDecMaxWg; ++w)
                if (w < a.n_wg) v += pv[w];
            for (int w = kDecMaxWg; w < a.n_wg; ++w)
                v += __builtin_nontemporal_load(&a.partial[((int64_t)w * kSmallT + t) * kDecE + ee]);
            float l = (float)v;
            if (a.bias) l = __fadd_rn(l, a.bias[ee]);
            lg[t][ee] = l;
        }
    }
    lds_barrier();
    // rank of expert e in its token's order (logit descending, id ascending):
    // the experts before e with a logit >= its own and those after it with a
    // larger one; rank < k selects it at slot rank.  A row holding a NaN
    // takes the sequential scan instead (its order is scan-dependent).
    if (tid < T * kDecE) {
        const int t = tid / kDecE, e = tid % kDecE;
        if (e < E) {
            const float le = lg[t][e];
            int r = 0;
            bool ordered = true;
            for (int q = 0; q < E; ++q) {
                const float lq = lg[t][q];
                ordered = ordered && lq == lq;
                r += q < e ? (lq >= le ? 1 : 0) : (lq > le ? 1 : 0);
            }
            s_rank[t][e] = ordered ? r : -1;
            if (ordered && r < k) s_ids[t * k + r] = e;
        }
    }
    lds_barrier();
    if (tid < T) {
        const int t = tid;
        if (s_rank[t][0] < 0) {
            select_token<kDecE>(&lg[t][0], E, k, &s_ids[t * k], &s_w[t * k]);
        } else {
            // weights in slot order, as the sequential selection forms them
            const float lmax = lg[t][s_ids[t * k]];
            float z = 0.f;
            for (int j2 = 0; j2 < k; ++j2) {
                const float p = expf(lg[t][s_ids[t * k + j2]] - lmax);
                s_w[t * k + j2] = p;
                z += p;
            }
            const float inv = 1.0f / z;
            for (int j2 = 0; j2 < k; ++j2) s_w[t * k + j2] = s_w[t * k + j2] * inv;
        }
    }
    lds_barrier();
    const int P = T * k;
    const int lo = a.e_begin, hi = a.e_begin + a.n_local;
    if (tid < E) {
        int c = 0;
        if (tid >= lo && tid < hi)
            for (int p = 0; p < P; ++p) c += (s_ids[p] == tid);
        s_cnt[tid] = c;
    }
    lds_barrier();
    // per expert: its first row, active-list slot and first tile, from
    // prefix sums over the experts before it (lanes 0..15 of wave 0)
    if (wid == 0) {
        const int c = tid < E ? s_cnt[tid] : 0;
        const int nz = c > 0 ? 1 : 0;
        const int tl = (c + a.tile_rows - 1) / a.tile_rows;
        int run = c, na = nz, nt = tl;
#pragma unroll
        for (int off = 1; off < kDecE; off <<= 1) {
            const int r1 = __shfl_up(run, off, 64), n1 = __shfl_up(na, off, 64),
                      t1 = __shfl_up(nt, off, 64);
            if (lane >= off) { run += r1; na += n1; nt += t1; }
        }
        run -= c; na -= nz; nt -= tl;   // exclusive
        if (tid < E) {
            s_off[tid] = run;
            a.rv.counts[tid] = c;
            a.rv.offsets[tid] = run;
            if (c > 0) {
                a.rv.active[1 + na] = tid;
                for (int r = 0; r < c; r += a.tile_rows) {
                    a.rv.tiles[2 * nt] = tid;
                    a.rv.tiles[2 * nt + 1] = run + r;
                    ++nt;
                }
            }
            if (tid == E - 1) {
                a.rv.offsets[E] = run + c;
                a.rv.active[0] = na + nz;
                *a.rv.n_tiles = nt;
            }
        }
    }
    lds_barrier();
    if (tid < P) {
        const int ee = s_ids[tid];
        a.rv.topk_idx[tid] = ee;
        a.rv.topk_w[tid] = s_w[tid];
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
    if (tid < T * kDecE) {
        const int t = tid / kDecE, ee = tid % kDecE;
        if (ee < E) a.rv.logits[(int64_t)t * E + ee] = lg[t][ee];
    }
}

// Router and selection for many tokens: 8 tokens per 256-thread workgroup;
// wave w takes tokens 4(w/2) .. +3 and experts 8(w%2) .. +7 (then +16, ...).
// Lane l accumulates, in fp64, the 8-element groups l, l + 64, ... of the
// reduction axis for its 4 tokens x 8 experts, so each router value it
// loads serves 4 tokens and each x value 8 experts, and a wave reads 512
// consecutive elements of every row per step (two steps in flight).  A
// fixed transpose-reduce over the 64 lanes sums the lane partials (32
// shuffles for the 32 sums); each sum is rounded once to fp32 and the bias
// added in fp32; then one thread per token selects its experts from the
// logits in LDS.
constexpr int kRsTokWave = 4;
constexpr int kRsExp = 8;
constexpr int kRsTok = 2 * kRsTokWave;
constexpr int kRsThreads = 4 * kWave;

__global__ __launch_bounds__(kRsThreads) void router_select_kernel(const uint16_t* __restrict__ x,
                                                                   const float* __restrict__ wrT,
                                                                   const float* __restrict__ bias,
                                                                   int T, int d, int E, int k,
                                                                   RouteView rv)
{
    __shared__ float lg[kRsTok][64];
    const int wid = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int tg = wid / 2, eh = wid % 2;
    const int t0 = blockIdx.x * kRsTok + tg * kRsTokWave;
    for (int e0 = eh * kRsExp; e0 < E; e0 += 2 * kRsExp) {
        double acc[kRsTokWave][kRsExp];
#pragma unroll
        for (int i = 0; i < kRsTokWave; ++i)
#pragma unroll
            for (int j = 0; j < kRsExp; ++j) acc[i][j] = 0.0;
        // tokens past T and experts past E (partial last groups) recompute
        // token T-1 / expert E-1 so that the loop has no branch; their sums
        // are dropped
        const uint16_t* xr[kRsTokWave];
        const float* wr[kRsExp];
#pragma unroll
        for (int i = 0; i < kRsTokWave; ++i) xr[i] = x + (int64_t)min(t0 + i, T - 1) * d;
#pragma unroll
        for (int j = 0; j < kRsExp; ++j) wr[j] = wrT + (int64_t)min(e0 + j, E - 1) * d;
        // two steps of loads in flight: step g + 512 is fetched while step g
        // computes (a prefetch past d re-reads the lane's current step)
        struct Step {
            u32x4_t xv[kRsTokWave];
            float4 w0[kRsExp], w1[kRsExp];
        };
        auto fetch = [&](Step& st, int g) {
#pragma unroll
            for (int i = 0; i < kRsTokWave; ++i) st.xv[i] = *reinterpret_cast<const u32x4_t*>(xr[i] + g);
#pragma unroll
            for (int j = 0; j < kRsExp; ++j) {
                st.w0[j] = *reinterpret_cast<const float4*>(wr[j] + g);
                st.w1[j] = *reinterpret_cast<const float4*>(wr[j] + g + 4);
            }
        };
        auto fma_step = [&](const Step& st) {
#pragma unroll
            for (int j = 0; j < kRsExp; ++j)
#pragma unroll
                for (int i = 0; i < kRsTokWave; ++i) fma8(acc[i][j], st.xv[i], st.w0[j], st.w1[j]);
        };
        constexpr int kStep = kWave * 8;
        Step s0, s1;
        int g = lane * 8;
        if (g < d) fetch(s0, g);
        for (; g < d; g += 2 * kStep) {
            const bool more = g + kStep < d;
            fetch(s1, more ? g + kStep : g);
            fma_step(s0);
            if (!more) break;
            const bool more2 = g + 2 * kStep < d;
            fetch(s0, more2 ? g + 2 * kStep : g);
            fma_step(s1);
        }
        // transpose-reduce over the 64 lanes: at the step with lane offset o
        // a lane keeps half of its n values (the upper half if its o bit is
        // set), sends the other half to lane ^ o and adds what it receives;
        // after offsets 32..2 each lane holds one value summed over 32 lanes,
        // and offset 1 completes it.  Value q = 8 i + j ends on the lanes whose
        // bits 5..1 spell q (bit 5 most significant).  Fixed order.
        constexpr int kVals = kRsTokWave * kRsExp;   // 32
        double v[kVals];
#pragma unroll
        for (int i = 0; i < kRsTokWave; ++i)
#pragma unroll
            for (int j = 0; j < kRsExp; ++j) v[i * kRsExp + j] = acc[i][j];
#pragma unroll
        for (int o = kWave / 2, n = kVals; o >= 2; o >>= 1, n >>= 1) {
            const bool up = (lane & o) != 0;
#pragma unroll
            for (int m = 0; m < kVals / 2; ++m) {
                if (m < n / 2) {
                    const double send = up ? v[m] : v[m + n / 2];
                    const double keep = up ? v[m + n / 2] : v[m];
                    v[m] = keep + __shfl_xor(send, o, kWave);
                }
            }
        }
        const double total = v[0] + __shfl_xor(v[0], 1, kWave);
        const int q = ((lane >> 5) & 1) * 16 + ((lane >> 4) & 1) * 8 + ((lane >> 3) & 1) * 4 +
                      ((lane >> 2) & 1) * 2 + ((lane >> 1) & 1);
        if ((lane & 1) == 0) {
            const int i = q / kRsExp, j = q % kRsExp;
            const int t = t0 + i, e = e0 + j;
            if (t < T && e < E) {
                float lv = (float)total;
                if (bias) lv = __fadd_rn(lv, bias[e]);
                lg[tg * kRsTokWave + i][e] = lv;
                rv.logits[(int64_t)t * E + e] = lv;
            }
        }
    }
    lds_barrier();
    if (threadIdx.x < kRsTok) {
        const int t = blockIdx.x * kRsTok + threadIdx.x;
        if (t < T) select_token_any(&lg[threadIdx.x][0], t, E, k, rv);
    }
}

// Selection from caller-supplied fp32 logits (copied into the routing
// view): one thread per token.
__global__ __launch_bounds__(256) void select_kernel(const float* __restrict__ logits_in, int T,
                                                     int E, int k, RouteView rv)
{
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= T) return;
    const float* l = logits_in + (int64_t)t * E;
    for (int e = 0; e < E; ++e) rv.logits[(int64_t)t * E + e] = l[e];
    select_token_any(l, t, E, k, rv);
}

// Expert-grouped permutation of the T*k pairs (one 1024-thread workgroup),
// rows grouped by local expert, then by pair (token, slot) order.
//  1. counts: LDS histogram of the local pairs (order-free); thread 0 then
//     writes counts, offsets, the active-expert list and the GEMM tile list.
//  2. rows: pairs in rounds of 1024 x 8; each thread holds 8 consecutive
//     pairs; per group of 16 experts, one wave scan of packed per-thread
//     counts plus a scan of the wave totals give each pair its row after the
//     expert's cursor.
// Deterministic: no atomic decides a row.
constexpr int kPermChunk = 8;
constexpr int kPermGroup = 16;   // experts counted together (packed counters)

struct PermArgs {
    int T, E, k, e_begin, n_local, tile_rows;
    RouteView rv;
};

__global__ __launch_bounds__(kRouteThreads) void permute_kernel(PermArgs a)
{
    constexpr int kWords = kPermGroup / 2;   // two 16-bit counters per word
    __shared__ int hist[64];
    __shared__ int cursor[64];
    __shared__ uint32_t wtot[kRouteWaves][kWords];
    __shared__ uint32_t wpre[kRouteWaves][kWords];
    __shared__ uint32_t rtot[kWords];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int E = a.E, k = a.k, P = a.T * a.k;
    const int lo = a.e_begin, hi = a.e_begin + a.n_local;
    const RouteView& rv = a.rv;
    if (tid < 64) hist[tid] = 0;
    lds_barrier();
    for (int p = tid; p < P; p += kRouteThreads) {
        const int e = rv.topk_idx[p];
        if (e >= lo && e < hi) atomicAdd(&hist[e], 1);
    }
    lds_barrier();
    // offsets, active list and tiles: prefix sums over the experts (wave 0)
    if (wid == 0) {
        int c = lane < E ? hist[lane] : 0;
        const int nz = c > 0 ? 1 : 0;
        const int tl = (c + a.tile_rows - 1) / a.tile_rows;
        int run = c, na = nz, nt = tl;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int r1 = __shfl_up(run, off, 64), n1 = __shfl_up(na, off, 64),
                      t1 = __shfl_up(nt, off, 64);
            if (lane >= off) { run += r1; na += n1; nt += t1; }
        }
        run -= c; na -= nz; nt -= tl;   // exclusive
        if (lane < E) {
            rv.counts[lane] = c;
            rv.offsets[lane] = run;
            cursor[lane] = run;
            if (c > 0) {
                rv.active[1 + na] = lane;
                for (int r = 0; r < c; r += a.tile_rows) {
                    rv.tiles[2 * nt] = lane;
                    rv.tiles[2 * nt + 1] = run + r;
                    ++nt;
                }
            }
            if (lane == E - 1) {
                rv.offsets[E] = run + c;
                rv.active[0] = na + nz;
                *rv.n_tiles = nt;
            }
        }
    }
    lds_barrier();
    // rows: rounds of 1024 x 8 pairs; thread t holds pairs 8t .. 8t+7 of the
    // round.  Per group of 16 experts, each thread packs its per-expert counts
    // two to a word (a round has at most 8192 pairs, below 2^16), one
    // wave-level scan and one scan over the wave totals give every thread the
    // rows of its pairs: cursor[e] + pairs of expert e in earlier threads +
    // earlier pairs of its own.
    for (int r0 = 0; r0 < P; r0 += kRouteThreads * kPermChunk) {
        const int p0 = r0 + tid * kPermChunk;
        int ids[kPermChunk];
#pragma unroll
        for (int q = 0; q < kPermChunk; ++q) {
            ids[q] = p0 + q < P ? rv.topk_idx[p0 + q] : -1;
            if (p0 + q < P && (ids[q] < lo || ids[q] >= hi)) rv.pair_row[p0 + q] = -1;
        }
        for (int g0 = lo - lo % kPermGroup; g0 < hi; g0 += kPermGroup) {
            uint32_t c[kWords];
#pragma unroll
            for (int m = 0; m < kWords; ++m) c[m] = 0u;
#pragma unroll
            for (int q = 0; q < kPermChunk; ++q) {
                const int rel = ids[q] - g0;
                const bool mine = ids[q] >= lo && ids[q] < hi && rel >= 0 && rel < kPermGroup;
#pragma unroll
                for (int m = 0; m < kWords; ++m)
                    if (mine && (rel >> 1) == m) c[m] += 1u << (16 * (rel & 1));
            }
            uint32_t inc[kWords];
#pragma unroll
            for (int m = 0; m < kWords; ++m) {
                uint32_t v = c[m];
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    const uint32_t o = __shfl_up(v, off, 64);
                    if (lane >= off) v += o;
                }
                inc[m] = v;
            }
            if (lane == 63) {
#pragma unroll
                for (int m = 0; m < kWords; ++m) wtot[wid][m] = inc[m];
            }
            lds_barrier();
            if (tid < kRouteWaves * kWords) {
                const int w = tid / kWords, m = tid % kWords;
                uint32_t pre = 0u;
                for (int w2 = 0; w2 < w; ++w2) pre += wtot[w2][m];
                wpre[w][m] = pre;
                if (w == kRouteWaves - 1) rtot[m] = pre + wtot[w][m];
            }
            lds_barrier();
            // exclusive count of each expert's pairs before this thread's
            uint32_t ex[kWords];
#pragma unroll
            for (int m = 0; m < kWords; ++m) ex[m] = wpre[wid][m] + inc[m] - c[m];
            uint32_t own[kWords];
#pragma unroll
            for (int m = 0; m < kWords; ++m) own[m] = 0u;
#pragma unroll
            for (int q = 0; q < kPermChunk; ++q) {
                const int rel = ids[q] - g0;
                const bool mine = ids[q] >= lo && ids[q] < hi && rel >= 0 && rel < kPermGroup;
                if (mine) {
                    uint32_t before = 0u;
#pragma unroll
                    for (int m = 0; m < kWords; ++m)
                        if ((rel >> 1) == m) {
                            const int sh = 16 * (rel & 1);
                            before = ((ex[m] >> sh) & 0xFFFFu) + ((own[m] >> sh) & 0xFFFFu);
                            own[m] += 1u << sh;
                        }
                    const int row = cursor[ids[q]] + (int)before;
                    rv.pair_row[p0 + q] = row;
                    rv.row_token[row] = (p0 + q) / k;
                }
            }
            lds_barrier();   // every thread has read cursor and wpre
            if (tid < kPermGroup && g0 + tid >= lo && g0 + tid < hi)
                cursor[g0 + tid] += (int)((rtot[tid >> 1] >> (16 * (tid & 1))) & 0xFFFFu);
            lds_barrier();
        }
    }
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

extern "C" int moe_route_decode_ok(int T, int E, int k)
{
    return T >= 1 && T <= moe::kSmallT && E <= moe::kDecE && T * k <= moe::kDecPairs;
}

extern "C" int moe_route_decode_wgs(int d) { return (d / 8 + 63) / 64; }



extern "C" hipError_t moe_launch_route_decode(const uint16_t* x, const float* wrT,
                                              const float* bias, double* partial, int T, int d,
                                              int E, int k, int e_begin, int n_local, int tile_rows,
                                              const moe::RouteView* rv, hipStream_t s)
{
    moe::DecodeRouteArgs a{};
    a.x = x; a.wrT = wrT; a.bias = bias; a.partial = partial;
    a.T = T; a.d = d; a.E = E; a.k = k;
    a.e_begin = e_begin; a.n_local = n_local; a.tile_rows = tile_rows;
    a.rv = *rv;
    a.n_wg = moe_route_decode_wgs(d);
    hipLaunchKernelGGL(moe::route_partials_kernel, dim3(a.n_wg), dim3(moe::kRouteThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(moe::route_finish_kernel, dim3(1), dim3(moe::kRouteThreads), 0, s, a);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_router_select(const uint16_t* x, const float* wrT,
                                               const float* bias, int T, int d, int E, int k,
                                               const moe::RouteView* rv, hipStream_t s)
{
    const int grid = (T + moe::kRsTok - 1) / moe::kRsTok;
    hipLaunchKernelGGL(moe::router_select_kernel, dim3(grid), dim3(moe::kRsThreads), 0, s, x, wrT,
                       bias, T, d, E, k, *rv);
    return hipGetLastError();
}

extern "C" hipError_t moe_launch_route(const float* logits_in, int T, int E, int k, int e_begin,
                                       int n_local, int tile_rows, const moe::RouteView* rv,
                                       hipStream_t s)
{
    if (logits_in) {
        hipLaunchKernelGGL(moe::select_kernel, dim3((T + 255) / 256), dim3(256), 0, s, logits_in, T,
                           E, k, *rv);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    moe::PermArgs a{};
    a.T = T; a.E = E; a.k = k;
    a.e_begin = e_begin; a.n_local = n_local; a.tile_rows = tile_rows;
    a.rv = *rv;
    hipLaunchKernelGGL(moe::permute_kernel, dim3(1), dim3(moe::kRouteThreads), 0, s, a);
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
