/*
 * moe_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU definition of one DBRX-style Mixture-of-Experts
 * layer, used by the test-suite, the smoke check and the CPU-baseline leg of
 * the benchmark to judge the GPU library.  Nothing in the product path may
 * link, load or call this file.  It shares no code with the GPU library.
 *
 * What the layer is (Chen et al., "Towards Building Private LLMs: Exploring
 * Multi-Node Expert Parallelism on Apple Silicon for Mixture-of-Experts Large
 * Language Model", RACS'24):
 *   - Sec. 2.1 (Mixture-of-Experts): the single FFN of a decoder block is
 *     replaced by 16 independent FFN experts; DBRX selects 4 of the 16 per
 *     token in every layer.
 *   - Sec. 2.2 (Parallelization Techniques, expert parallelism): once the
 *     router-selected experts have run, their outputs are combined by a
 *     weighted sum.
 *   - Sec. 3.1 (fork-join figure): the router output decides which experts
 *     (and therefore which nodes) receive a token.
 *   - Table tab:vars, note (e): each expert has three matrices v1, w1, w2 of
 *     size D_embed x D_ffn.
 *   - Sec. 4.2 (Busy Full Loading): evaluating every expert and zeroing the
 *     unselected ones in the weighted sum gives the same result; that dense
 *     form is oracle_layer_dense() below.
 *
 * Readings where the paper is silent (R1..R8):
 *   R1 router = one linear map, fp32 weights [d,E]; logit = fp32 rounding of
 *      the exact dot product, then an optional fp32 bias is added in fp32.
 *   R2 selection by logit, ties to the lower expert id, slots ordered by
 *      (logit desc, id asc); +0 and -0 compare equal.
 *   R3 gate weights = softmax of the selected logits (renormalised top-k).
 *   R4 w1 is the gate (SiLU applied), v1 the up projection, w2 the down one;
 *      silu(z) = z * sigmoid(z).
 *   R5 bf16 (round-to-nearest-even) only at the inputs, at H (the operand of
 *      the down projection) and at the layer output y.
 *   R6 the routing weight multiplies the expert output after the down
 *      projection; the combine sums local slots in slot order.
 *   R7 an expert-parallel share [e_begin, e_begin+n_local) keeps the routing
 *      of the full layer and sums only its local slots (no renormalisation).
 *   R8 rows of the permutation are grouped by expert ascending, then token
 *      ascending.
 *
 * Tensor layouts at this interface (all row-major):
 *   x      bf16 bits [T, d]          router wr fp32 [d, E], bias fp32 [E]
 *   gate   bf16 bits [d, f]  (w1)    up bf16 bits [d, f] (v1)
 *   down   bf16 bits [f, d]  (w2)    y  bf16 bits [T, d]
 * Per-expert weights are passed as arrays of E pointers; an entry may be NULL
 * only if that expert is never used by the call.
 *
 * Every sum is accumulated in fp64 in increasing index order, so results do
 * not depend on the OpenMP thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EARG (-1)

/* ---------------------------------------------------------------- bf16 -- */

/* bf16 bits -> double, exact (bf16 is the top half of an fp32). */
double oracle_f64_from_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* double -> bf16 bits, one rounding, round-to-nearest-even (R5).
 * The value is scaled by the bf16 quantum at its binade (fixed at 2^-133 in
 * the subnormal range), rounded to an integer with rint() in the default
 * rounding mode (nearest-even), and scaled back.  All scalings are by powers
 * of two and therefore exact. */
uint16_t oracle_bf16_from_f64(double v)
{
    if (isnan(v))
        return signbit(v) ? 0xFFC0u : 0x7FC0u;
    uint16_t sign = signbit(v) ? 0x8000u : 0u;
    double a = fabs(v);
    if (a == 0.0)
        return sign;
    if (isinf(a))
        return (uint16_t)(sign | 0x7F80u);
    int e2;
    (void)frexp(a, &e2);           /* a in [2^(e2-1), 2^e2) */
    int lead = e2 - 1;
    if (lead < -126)
        lead = -126;               /* subnormal bf16: fixed quantum */
    double q = ldexp(1.0, lead - 7);
    double r = rint(a / q) * q;
    if (r >= 0x1.0p128)
        return (uint16_t)(sign | 0x7F80u);
    float f = (float)r;            /* exact: r has at most 8 significant bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(sign | (uint16_t)(u >> 16));
}

void oracle_bf16_round_array(const double *in, uint16_t *out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_bf16_from_f64(in[i]);
}

/* -------------------------------------------------------------- router -- */

/* R1: logits[t,e] = fp32( sum_i x[t,i]*wr[i,e] ), then + bias[e] in fp32. */
int oracle_router_logits(int T, int d, int E, const uint16_t *x,
                         const float *wr, const float *bias, float *logits)
{
    if (T < 0 || d <= 0 || E <= 0 || (T > 0 && (!x || !wr || !logits)))
        return ORC_EARG;
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t) {
        for (int e = 0; e < E; ++e) {
            double s = 0.0;
            for (int i = 0; i < d; ++i)
                s += oracle_f64_from_bf16(x[(int64_t)t * d + i]) * (double)wr[(int64_t)i * E + e];
            float l = (float)s;
            if (bias) {
                volatile float lb = l + bias[e];   /* fp32 add, one rounding */
                l = lb;
            }
            logits[(int64_t)t * E + e] = l;
        }
    }
    return ORC_OK;
}

/* R2 + R3 on given fp32 logits.  idx[t,j] = expert id of slot j, w[t,j] =
 * exp(l_j - l_max) / sum_j' exp(l_j' - l_max) over the selected slots. */
int oracle_route_from_logits(int T, int E, int k, const float *logits,
                             int32_t *idx, double *w)
{
    if (T < 0 || E <= 0 || k <= 0 || k > E || (T > 0 && (!logits || !idx || !w)))
        return ORC_EARG;
    for (int t = 0; t < T; ++t) {
        const float *l = logits + (int64_t)t * E;
        for (int e = 0; e < E; ++e)
            if (!isfinite(l[e]))
                return ORC_EARG;
        unsigned char taken[256];
        if (E > 256)
            return ORC_EARG;
        memset(taken, 0, sizeof taken);
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                if (taken[e])
                    continue;
                /* strict '>' over increasing e: equal logits keep the lower id */
                if (best < 0 || l[e] > l[best])
                    best = e;
            }
            taken[best] = 1;
            idx[(int64_t)t * k + j] = best;
        }
        double lmax = (double)l[idx[(int64_t)t * k]];
        double z = 0.0;
        for (int j = 0; j < k; ++j)
            z += exp((double)l[idx[(int64_t)t * k + j]] - lmax);
        for (int j = 0; j < k; ++j)
            w[(int64_t)t * k + j] = exp((double)l[idx[(int64_t)t * k + j]] - lmax) / z;
    }
    return ORC_OK;
}

/* --------------------------------------------------------- permutation -- */

/* R8: counts[e] = #pairs routed to local expert e (0 for non-local experts),
 * offsets = exclusive prefix sum of counts (E+1 entries), pair_row[t*k+j] =
 * row of pair (t,j) in the expert-grouped order, or -1 if its expert is not
 * local; row_token[r] = token of row r. */
int oracle_permutation(int T, int E, int k, int e_begin, int n_local,
                       const int32_t *idx, int32_t *counts, int32_t *offsets,
                       int32_t *pair_row, int32_t *row_token)
{
    if (T < 0 || E <= 0 || k <= 0 || e_begin < 0 || n_local <= 0 ||
        e_begin + n_local > E || !counts || !offsets)
        return ORC_EARG;
    for (int e = 0; e < E; ++e)
        counts[e] = 0;
    for (int64_t p = 0; p < (int64_t)T * k; ++p) {
        int e = idx[p];
        if (e < 0 || e >= E)
            return ORC_EARG;
        if (e >= e_begin && e < e_begin + n_local)
            counts[e]++;
    }
    offsets[0] = 0;
    for (int e = 0; e < E; ++e)
        offsets[e + 1] = offsets[e] + counts[e];
    int32_t *fill = (int32_t *)calloc((size_t)E, sizeof(int32_t));
    if (!fill)
        return ORC_EARG;
    for (int t = 0; t < T; ++t) {           /* tokens in increasing order */
        for (int j = 0; j < k; ++j) {
            int e = idx[(int64_t)t * k + j];
            if (e >= e_begin && e < e_begin + n_local) {
                int r = offsets[e] + fill[e]++;
                pair_row[(int64_t)t * k + j] = r;
                row_token[r] = t;
            } else {
                pair_row[(int64_t)t * k + j] = -1;
            }
        }
    }
    free(fill);
    return ORC_OK;
}

/* ---------------------------------------------------------- expert GLU -- */

static double silu(double z)
{
    /* z * sigmoid(z), written so that neither branch overflows */
    if (z >= 0.0)
        return z / (1.0 + exp(-z));
    double ez = exp(z);
    return z * ez / (1.0 + ez);
}

/* One expert on m rows (R4, R5):
 *   g = x w1, u = x v1 (fp64), h = silu(g) * u, hb = bf16(h), o = hb w2 (fp64).
 * xrows bf16 [m,d]; hb_out bf16 [m,f] (may be NULL); o_out fp64 [m,d].
 * round_h = 0 is the information-only exact form: the down projection takes
 * h itself instead of hb (hb_out still receives bf16(h)). */
static int expert_glu(int m, int d, int f, const uint16_t *xrows,
                      const uint16_t *gate, const uint16_t *up,
                      const uint16_t *down, int round_h, uint16_t *hb_out, double *o_out)
{
    if (m < 0 || d <= 0 || f <= 0 || (m > 0 && (!xrows || !gate || !up || !down || !o_out)))
        return ORC_EARG;
    double *g = (double *)malloc(sizeof(double) * (size_t)f);
    double *u = (double *)malloc(sizeof(double) * (size_t)f);
    double *hb = (double *)malloc(sizeof(double) * (size_t)f);
    if (!g || !u || !hb) {
        free(g); free(u); free(hb);
        return ORC_EARG;
    }
    for (int r = 0; r < m; ++r) {
        const uint16_t *xr = xrows + (int64_t)r * d;
        /* gate/up: each column n sums over i = 0..d-1 in order */
#pragma omp parallel for schedule(static)
        for (int n0 = 0; n0 < f; n0 += 256) {
            int n1 = n0 + 256 < f ? n0 + 256 : f;
            for (int n = n0; n < n1; ++n) {
                g[n] = 0.0;
                u[n] = 0.0;
            }
            for (int i = 0; i < d; ++i) {
                double xi = oracle_f64_from_bf16(xr[i]);
                const uint16_t *gw = gate + (int64_t)i * f;
                const uint16_t *uw = up + (int64_t)i * f;
                for (int n = n0; n < n1; ++n) {
                    g[n] += xi * oracle_f64_from_bf16(gw[n]);
                    u[n] += xi * oracle_f64_from_bf16(uw[n]);
                }
            }
            for (int n = n0; n < n1; ++n) {
                double h = silu(g[n]) * u[n];
                uint16_t hbits = oracle_bf16_from_f64(h);
                hb[n] = round_h ? oracle_f64_from_bf16(hbits) : h;
                if (hb_out)
                    hb_out[(int64_t)r * f + n] = hbits;
            }
        }
        /* down: each output column n sums over j = 0..f-1 in order */
        double *orow = o_out + (int64_t)r * d;
#pragma omp parallel for schedule(static)
        for (int n0 = 0; n0 < d; n0 += 256) {
            int n1 = n0 + 256 < d ? n0 + 256 : d;
            for (int n = n0; n < n1; ++n)
                orow[n] = 0.0;
            for (int j = 0; j < f; ++j) {
                double hj = hb[j];
                const uint16_t *dw = down + (int64_t)j * d;
                for (int n = n0; n < n1; ++n)
                    orow[n] += hj * oracle_f64_from_bf16(dw[n]);
            }
        }
    }
    free(g); free(u); free(hb);
    return ORC_OK;
}

int oracle_expert_glu(int m, int d, int f, const uint16_t *xrows,
                      const uint16_t *gate, const uint16_t *up,
                      const uint16_t *down, uint16_t *hb_out, double *o_out)
{
    return expert_glu(m, d, f, xrows, gate, up, down, 1, hb_out, o_out);
}

/* ---------------------------------------------------------------- layer -- */

/* Steps 4-5 of the layer on a given routing (R6, R7):
 *   y[t] = bf16( sum over slots j of t whose expert is local: w[t,j] * o_j ).
 * y64 (fp64 [T,d], before the final rounding), y16 (bf16 [T,d]) and hb
 * (bf16 [T*k, f]: row t*k+j receives pair (t,j)'s hb when its expert is
 * local; other rows are left as they are) may each be NULL.  round_h = 0 is
 * the information-only exact form (no rounding of H; y64 is then the layer
 * with no intermediate rounding at all). */
int oracle_layer_with_routing_ex(int T, int d, int f, int E, int k, int e_begin,
                                 int n_local, const uint16_t *x, const int32_t *idx,
                                 const double *w, const uint16_t *const *gate,
                                 const uint16_t *const *up,
                                 const uint16_t *const *down, int round_h, double *y64,
                                 uint16_t *y16, uint16_t *hb)
{
    if (T < 0 || d <= 0 || f <= 0 || E <= 0 || k <= 0 || k > E || e_begin < 0 ||
        n_local <= 0 || e_begin + n_local > E)
        return ORC_EARG;
    double *o = (double *)malloc(sizeof(double) * (size_t)d);
    double *acc = (double *)malloc(sizeof(double) * (size_t)d);
    if (!o || !acc) {
        free(o); free(acc);
        return ORC_EARG;
    }
    int rc = ORC_OK;
    for (int t = 0; t < T && rc == ORC_OK; ++t) {
        for (int n = 0; n < d; ++n)
            acc[n] = 0.0;
        for (int j = 0; j < k; ++j) {            /* slot order */
            int e = idx[(int64_t)t * k + j];
            if (e < 0 || e >= E) { rc = ORC_EARG; break; }
            if (e < e_begin || e >= e_begin + n_local)
                continue;
            if (!gate[e] || !up[e] || !down[e]) { rc = ORC_EARG; break; }
            rc = expert_glu(1, d, f, x + (int64_t)t * d, gate[e], up[e], down[e], round_h,
                            hb ? hb + ((int64_t)t * k + j) * f : NULL, o);
            if (rc != ORC_OK)
                break;
            double wj = w[(int64_t)t * k + j];
            for (int n = 0; n < d; ++n)
                acc[n] += wj * o[n];
        }
        for (int n = 0; n < d; ++n) {
            if (y64)
                y64[(int64_t)t * d + n] = acc[n];
            if (y16)
                y16[(int64_t)t * d + n] = oracle_bf16_from_f64(acc[n]);
        }
    }
    free(o); free(acc);
    return rc;
}

int oracle_layer_with_routing(int T, int d, int f, int E, int k, int e_begin,
                              int n_local, const uint16_t *x, const int32_t *idx,
                              const double *w, const uint16_t *const *gate,
                              const uint16_t *const *up,
                              const uint16_t *const *down, double *y64,
                              uint16_t *y16)
{
    return oracle_layer_with_routing_ex(T, d, f, E, k, e_begin, n_local, x, idx, w, gate, up,
                                        down, 1, y64, y16, NULL);
}

/* The whole layer: router logits, selection and weights, then the experts
 * and the weighted combine.  logits/idx/w outputs may be NULL. */
int oracle_layer(int T, int d, int f, int E, int k, int e_begin, int n_local,
                 const uint16_t *x, const float *wr, const float *bias,
                 const uint16_t *const *gate, const uint16_t *const *up,
                 const uint16_t *const *down, float *logits_out,
                 int32_t *idx_out, double *w_out, double *y64, uint16_t *y16)
{
    if (T < 0 || E <= 0 || k <= 0 || k > E)
        return ORC_EARG;
    size_t nT = (size_t)(T > 0 ? T : 1);
    float *lg = logits_out ? logits_out : (float *)malloc(sizeof(float) * nT * (size_t)E);
    int32_t *ix = idx_out ? idx_out : (int32_t *)malloc(sizeof(int32_t) * nT * (size_t)k);
    double *ww = w_out ? w_out : (double *)malloc(sizeof(double) * nT * (size_t)k);
    int rc = (!lg || !ix || !ww) ? ORC_EARG : ORC_OK;
    if (rc == ORC_OK)
        rc = oracle_router_logits(T, d, E, x, wr, bias, lg);
    if (rc == ORC_OK)
        rc = oracle_route_from_logits(T, E, k, lg, ix, ww);
    if (rc == ORC_OK)
        rc = oracle_layer_with_routing(T, d, f, E, k, e_begin, n_local, x, ix, ww,
                                       gate, up, down, y64, y16);
    if (!logits_out) free(lg);
    if (!idx_out) free(ix);
    if (!w_out) free(ww);
    return rc;
}

/* Busy-full-loading form (Sec. 4.2): every expert evaluates every token and
 * the unselected outputs are multiplied by zero in the weighted sum, which
 * runs over experts in id order.  Mathematically equal to the sparse layer;
 * y64 agrees with oracle_layer_with_routing to fp64 rounding. */
int oracle_layer_dense(int T, int d, int f, int E, int k, const uint16_t *x,
                       const int32_t *idx, const double *w,
                       const uint16_t *const *gate, const uint16_t *const *up,
                       const uint16_t *const *down, double *y64)
{
    if (T < 0 || d <= 0 || f <= 0 || E <= 0 || k <= 0 || k > E || !y64)
        return ORC_EARG;
    double *o = (double *)malloc(sizeof(double) * (size_t)d);
    double *wfull = (double *)malloc(sizeof(double) * (size_t)E);
    if (!o || !wfull) {
        free(o); free(wfull);
        return ORC_EARG;
    }
    int rc = ORC_OK;
    for (int t = 0; t < T && rc == ORC_OK; ++t) {
        for (int e = 0; e < E; ++e)
            wfull[e] = 0.0;
        for (int j = 0; j < k; ++j)
            wfull[idx[(int64_t)t * k + j]] = w[(int64_t)t * k + j];
        double *yr = y64 + (int64_t)t * d;
        for (int n = 0; n < d; ++n)
            yr[n] = 0.0;
        for (int e = 0; e < E; ++e) {
            rc = oracle_expert_glu(1, d, f, x + (int64_t)t * d, gate[e], up[e],
                                   down[e], NULL, o);
            if (rc != ORC_OK)
                break;
            for (int n = 0; n < d; ++n)
                yr[n] += wfull[e] * o[n];
        }
    }
    free(o); free(wfull);
    return rc;
}

/* Layer chaining for the stacked decode: x_next = bf16(x + y).  The sum of
 * two bf16 values is exact in fp64, so this is a single rounding. */
void oracle_residual_add(const uint16_t *x, const uint16_t *y, uint16_t *out,
                         int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_bf16_from_f64(oracle_f64_from_bf16(x[i]) +
                                      oracle_f64_from_bf16(y[i]));
}
