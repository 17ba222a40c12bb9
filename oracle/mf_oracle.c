/*
 * CPU oracle for the MeanField joint-configuration search.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header, table or helper with the
 * HIP library; the two meet only in the arrays the seeded generator draws.
 *
 * What it computes (plain definitions, written out):
 *   Joint space (Section II, Eq. 1): Lambda = prod_i Lambda_i.  A joint
 *     configuration is a linear index in lexicographic order, model 0 most
 *     significant (the order of itertools.product).
 *   Aggregate state (Section II, Eq. 2; Section III-B): the surrogate of model
 *     i sees its own option row plus an aggregate field summarising the
 *     combined resource pressure of all co-runners.  Here slot k of the
 *     aggregate is the sum, over all N models (model i included), of option
 *     column agg_cols[k] of the option each model runs.
 *   Surrogate (Section III-B, Eq. 6): one MLP g_i per model,
 *     (lat_i, thr_i) = W3 relu(W2 relu(W1 z + b1) + b2) + b3, z = [x_i | a].
 *   Constraints (Section II, Eq. 4 and the text after it): VRAM sum <= cap
 *     (inclusive) and a per-model latency bound lat_i <= sla_i (inclusive);
 *     any violation gives J = -inf.
 *   Decision (Section II): lambda* = argmax J; here J = sum_i omega_i thr_i,
 *     ties broken to the lowest linear index, top-k sorted by (J desc,
 *     index asc).
 *   Fixed observed state (Section III-B, the paper's own semantics, when
 *     fixed_state is given): the surrogate's aggregate input is the observed
 *     state, held fixed over the whole search, so model i's prediction
 *     depends on its own option only; the VRAM constraint still sums the
 *     candidate's options.
 *   Full utility (Section II, Eq. 3, when an objective block is given): with
 *     v the variant of model i's option, the normalised throughput is
 *     f_i = (thr_i - fmin_{i,v}) / (fmax_{i,v} - fmin_{i,v}) (per-variant
 *     min-max scaling); J = sum_i omega_i Q_{i,v} f_i
 *     - alpha sum_i eta_i c_i - beta sum_i max(0, tau_i + delta - f_i)^2,
 *     eta_i = 1 when model i changes variant from the previous step; the
 *     floor f_i >= tau_i joins the hard constraints (constraint after Eq. 3).
 *     Each model's term is evaluated in fp64 in this order: Rg = fmax - fmin,
 *     f = (thr - fmin) / Rg, q = Q f, J = fma(omega, q, J), J = J - alpha c
 *     (variant changed), d = (tau + delta) - f, J = J - beta (d d) if d > 0.
 *
 *   Output activation (Section III-B: the predictor ends in a sigmoid, when
 *     the sigmoid flag is set): lat = s(y0), thr = s(y1) with
 *     s(y) = 1 / (1 + e^-y), y clamped to [-700, 700] first.  e^x is defined
 *     by this algorithm (so that it is one function on every machine):
 *     k = rint(x * (1/ln 2)); r = x - k ln2_hi - k ln2_lo (two fmas, ln2_hi
 *     = ln 2 rounded to 24 bits); e^r by its Taylor series to degree 13
 *     (Horner, coefficients 1/n! rounded once, fma); times 2^k.
 *
 * Precision: every floating-point step is fp64.  Each dot product is one
 * fused multiply-add chain in ascending input order, starting from the bias;
 * relu(x) = (x > 0 ? x : +0).  The aggregate is summed in fp32 (model order)
 * and the oracle checks it against the fp64 sum: the generator's 2**-14 grid
 * makes them equal.  In bf16 mode the weights hold bfloat16 values and the
 * first hidden layer (the operand of the bf16 contraction) is quantised to
 * bfloat16: its pre-activation is accumulated in fp32 (the precision of the
 * contraction's accumulator: one fmaf chain in input order from the bias),
 * then relu, then rounded to bfloat16, ties to even; layers 2 and 3 stay fp64.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -march=x86-64-v3 -shared -fPIC.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#include "mf_oracle.h"

/* ---------------------------------------------------------------- helpers */

static int64_t stride_of(const orc_instance *in)
{
    int64_t nin = in->n_local + in->n_agg;
    return (int64_t)in->hidden1 * nin + in->hidden1 + (int64_t)in->hidden2 * in->hidden1 +
           in->hidden2 + 2 * in->hidden2 + 2;
}

/* Nearest bfloat16 value (8 significant bits), ties to even; x finite. */
static double bf16_round(double x)
{
    if (x == 0.0) return x;
    int e;
    frexp(fabs(x), &e);                 /* |x| = m * 2^e, m in [0.5, 1) */
    if (e < -125) e = -125;             /* bf16 subnormal spacing 2^-133 */
    double scale = ldexp(1.0, 8 - e);   /* |x| * scale in [128, 256) */
    return nearbyint(x * scale) / scale;
}

uint64_t orc_space_size(const orc_instance *in)
{
    uint64_t s = 1;
    for (int i = 0; i < in->n_models; i++) {
        uint64_t k = (uint64_t)in->n_options[i];
        if (k == 0) return 0;
        if (s > UINT64_MAX / k) return 0;   /* does not fit */
        s *= k;
    }
    return s;
}

/* Eq. 1: mixed-radix digits, model N-1 least significant. */
void orc_decode(const orc_instance *in, uint64_t idx, int32_t *digits)
{
    for (int i = in->n_models - 1; i >= 0; i--) {
        uint64_t k = (uint64_t)in->n_options[i];
        digits[i] = (int32_t)(idx % k);
        idx /= k;
    }
}

uint64_t orc_encode(const orc_instance *in, const int32_t *digits)
{
    uint64_t idx = 0;
    for (int i = 0; i < in->n_models; i++) idx = idx * (uint64_t)in->n_options[i] + (uint64_t)digits[i];
    return idx;
}

/* Aggregate field: slot k = sum over all models of column agg_cols[k] of the
 * chosen option row.  Returns 1 when the fp32 sum equals the fp64 sum. */
int orc_aggregate(const orc_instance *in, const int32_t *digits, float *a)
{
    int exact = 1;
    for (int k = 0; k < in->n_agg; k++) {
        float s32 = 0.0f;
        double s64 = 0.0;
        int64_t off = 0;
        for (int i = 0; i < in->n_models; i++) {
            float v = in->features[(off + digits[i]) * in->n_local + in->agg_cols[k]];
            s32 = s32 + v;
            s64 = s64 + (double)v;
            off += in->n_options[i];
        }
        a[k] = s32;
        if ((double)s32 != s64) exact = 0;
    }
    return exact;
}

/* One model's surrogate, canonical fp64.  w: fp64 copy of that model's packed
 * weights.  z: [L + A] inputs.  y[0] latency, y[1] throughput. */
/* e^x for |x| <= 700 (see the header comment for the definition). */
double orc_exp(double x)
{
    const double inv_ln2 = 1.4426950408889634;          /* 1 / ln 2 */
    const double ln2_hi = 0.693147182464599609375;      /* ln 2 to 24 significant bits */
    const double ln2_lo = -1.904654299957768e-09;       /* ln 2 - ln2_hi */
    const double k = rint(x * inv_ln2);
    double r = fma(-k, ln2_hi, x);
    r = fma(-k, ln2_lo, r);
    double fact = 1.0;
    double inv_fact[14];
    for (int n = 0; n < 14; n++) {
        if (n > 0) fact *= (double)n;
        inv_fact[n] = 1.0 / fact;
    }
    double p = inv_fact[13];
    for (int n = 12; n >= 0; n--) p = fma(p, r, inv_fact[n]);
    return ldexp(p, (int)k);
}

double orc_sigmoid(double y)
{
    const double c = y < -700.0 ? -700.0 : (y > 700.0 ? 700.0 : y);
    return 1.0 / (1.0 + orc_exp(-c));
}

static void mlp_forward(const double *w, int nin, int h1n, int h2n, int bf16, int sigmoid,
                        const double *z, double *h1, double *h2, double *y)
{
    const double *W1 = w, *b1 = W1 + (int64_t)h1n * nin, *W2 = b1 + h1n,
                 *b2 = W2 + (int64_t)h2n * h1n, *W3 = b2 + h2n, *b3 = W3 + 2 * h2n;
    for (int u = 0; u < h1n; u++) {
        if (bf16) {
            /* the bf16 layer-1 activation is a quantisation decided in the
             * precision the contraction accumulates in: fp32, one fused
             * multiply-add chain in input order from the bias */
            float c = (float)b1[u];
            for (int k = 0; k < nin; k++) c = fmaf((float)W1[(int64_t)u * nin + k], (float)z[k], c);
            c = c > 0.0f ? c : 0.0f;
            h1[u] = bf16_round((double)c);
        } else {
            double c = b1[u];
            for (int k = 0; k < nin; k++) c = fma(W1[(int64_t)u * nin + k], z[k], c);
            h1[u] = c > 0.0 ? c : 0.0;
        }
    }
    for (int v = 0; v < h2n; v++) {
        double c = b2[v];
        for (int u = 0; u < h1n; u++) c = fma(W2[(int64_t)v * h1n + u], h1[u], c);
        h2[v] = c > 0.0 ? c : 0.0;
    }
    for (int o = 0; o < 2; o++) {
        double c = b3[o];
        for (int v = 0; v < h2n; v++) c = fma(W3[(int64_t)o * h2n + v], h2[v], c);
        y[o] = sigmoid ? orc_sigmoid(c) : c;
    }
}

double *orc_weights_f64(const orc_instance *in)
{
    int64_t n = stride_of(in) * in->n_models;
    double *w = (double *)malloc(sizeof(double) * (size_t)n);
    if (!w) return NULL;
    for (int64_t t = 0; t < n; t++) w[t] = (double)in->weights[t];
    return w;
}

/* Full evaluation of one joint configuration.
 * flags: bit0 VRAM ok, bit1 every service constraint met (latency bounds;
 *        with an objective block also the throughput floors), bit2 feasible,
 *        bit3 aggregate exact; bit (8+i): model i misses one of them. */
void orc_eval_w(const orc_instance *in, const double *w64, uint64_t idx,
                     const float *sla, const float *omega, double *lat, double *thr,
                     double *J, uint32_t *flags, double *scratch)
{
    const int N = in->n_models, L = in->n_local, A = in->n_agg, nin = L + A;
    const int64_t stride = stride_of(in);
    int32_t d[ORC_MAX_MODELS];
    float a[ORC_MAX_AGG];
    double *z = scratch, *h1 = z + nin, *h2 = h1 + in->hidden1;
    orc_decode(in, idx, d);
    int exact = orc_aggregate(in, d, a);
    int vram_ok = (double)a[in->vram_slot] <= (double)in->vram_cap;
    int sla_ok = 1;
    uint32_t f = 0;
    int64_t off = 0;
    for (int i = 0; i < N; i++) {
        const float *x = in->features + (off + d[i]) * L;
        for (int k = 0; k < L; k++) z[k] = (double)x[k];
        for (int k = 0; k < A; k++) z[L + k] = (double)(in->fixed_state ? in->fixed_state[k] : a[k]);
        double y[2];
        mlp_forward(w64 + stride * i, nin, in->hidden1, in->hidden2, in->bf16, in->sigmoid, z, h1, h2, y);
        lat[i] = y[0];
        thr[i] = y[1];
        if (!(y[0] <= (double)sla[i])) { sla_ok = 0; f |= 1u << (8 + i); }
        off += in->n_options[i];
    }
    const orc_objective *ob = in->obj;
    double jq = 0.0;   /* Eq. 3 utility, model by model */
    if (ob) {
        int64_t row0 = 0;
        for (int i = 0; i < N; i++) {
            const int v = ob->variant[row0 + d[i]];
            const double fmin = (double)ob->fmin[i * ORC_MAX_VARIANTS + v];
            const double rg = (double)ob->fmax[i * ORC_MAX_VARIANTS + v] - fmin;
            const double fn = (thr[i] - fmin) / rg;                  /* per-variant min-max scaling */
            if (!(fn >= (double)ob->tau[i])) { sla_ok = 0; f |= 1u << (8 + i); }   /* throughput floor */
            const double q = (double)ob->quality[i * ORC_MAX_VARIANTS + v] * fn;
            jq = fma((double)omega[i], q, jq);
            if (ob->prev_variant[i] >= 0 && v != ob->prev_variant[i])       /* eta_i = 1: reload */
                jq = jq - (double)ob->alpha * (double)ob->reload_cost[i];
            const double dd = ((double)ob->tau[i] + (double)ob->delta) - fn;
            if (dd > 0.0) jq = jq - (double)ob->beta * (dd * dd);     /* soft SLA penalty */
            row0 += in->n_options[i];
        }
    }
    int feas = vram_ok && sla_ok;
    double j = -INFINITY;
    if (feas || in->raw_J) {
        if (ob) {
            j = jq;
        } else {
            j = 0.0;
            for (int i = 0; i < N; i++) j = fma((double)omega[i], thr[i], j);
        }
    }
    f |= (uint32_t)vram_ok | ((uint32_t)sla_ok << 1) | ((uint32_t)feas << 2) | ((uint32_t)exact << 3);
    *J = j;
    *flags = f;
}

size_t orc_scratch_doubles(const orc_instance *in)
{
    return (size_t)(in->n_local + in->n_agg + in->hidden1 + in->hidden2);
}

int orc_eval(const orc_instance *in, uint64_t idx, const float *sla, const float *omega,
             double *lat, double *thr, double *J, uint32_t *flags)
{
    double *w64 = orc_weights_f64(in);
    double *scr = (double *)malloc(sizeof(double) * orc_scratch_doubles(in));
    if (!w64 || !scr) { free(w64); free(scr); return -1; }
    orc_eval_w(in, w64, idx, sla, omega, lat, thr, J, flags, scr);
    free(w64);
    free(scr);
    return 0;
}

/* (J desc, idx asc) */
static int better(double ja, uint64_t ia, double jb, uint64_t ib)
{
    return ja > jb || (ja == jb && ia < ib);
}

static void topk_insert(double *tj, uint64_t *ti, int *cnt, int k, double j, uint64_t idx)
{
    if (*cnt == k && !better(j, idx, tj[k - 1], ti[k - 1])) return;
    int p = (*cnt < k) ? (*cnt)++ : k - 1;
    while (p > 0 && better(j, idx, tj[p - 1], ti[p - 1])) {
        tj[p] = tj[p - 1];
        ti[p] = ti[p - 1];
        p--;
    }
    tj[p] = j;
    ti[p] = idx;
}

/* Brute force over [lo, hi).  flag_dump: (hi-lo) x uint32 flags or NULL.
 * pred_dump: (hi-lo) x N x 2 doubles (lat, thr) or NULL.
 * J_dump: (hi-lo) doubles or NULL.  Returns 0, or -1 on bad arguments. */
int orc_search(const orc_instance *in, uint64_t lo, uint64_t hi, const float *sla,
               const float *omega, int k, int nthreads, orc_result *out,
               uint32_t *flag_dump, double *pred_dump, double *J_dump)
{
    const int N = in->n_models;
    uint64_t size = orc_space_size(in);
    if (N < 1 || N > ORC_MAX_MODELS || in->n_agg > ORC_MAX_AGG || k < 1 || k > ORC_MAX_TOPK ||
        size == 0 || lo > hi || hi > size)
        return -1;
    double *w64 = orc_weights_f64(in);
    if (!w64) return -1;
    memset(out, 0, sizeof(*out));
    const double bands[4] = {1e-5, 1e-4, 1e-3, 2e-2};
    double gJ[ORC_MAX_TOPK];
    uint64_t gI[ORC_MAX_TOPK];
    int gcnt = 0;
    uint64_t n_vram = 0, n_feas = 0, n_inexact = 0, near[4] = {0, 0, 0, 0};
    const int64_t n = (int64_t)(hi - lo);
    if (nthreads < 1) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads)
    {
        double tj[ORC_MAX_TOPK];
        uint64_t ti[ORC_MAX_TOPK];
        int tcnt = 0;
        uint64_t lv = 0, lf = 0, lx = 0, ln[4] = {0, 0, 0, 0};
        double lat[ORC_MAX_MODELS], thr[ORC_MAX_MODELS];
        double *scr = (double *)malloc(sizeof(double) * orc_scratch_doubles(in));
#pragma omp for schedule(static)
        for (int64_t t = 0; t < n; t++) {
            uint64_t idx = lo + (uint64_t)t;
            double J;
            uint32_t f;
            orc_eval_w(in, w64, idx, sla, omega, lat, thr, &J, &f, scr);
            lv += f & 1u;
            lf += (f >> 2) & 1u;
            lx += ((f >> 3) & 1u) ^ 1u;
            for (int i = 0; i < N; i++) {
                double dlt = fabs(lat[i] - (double)sla[i]);
                for (int b = 0; b < 4; b++) ln[b] += dlt <= bands[b];
            }
            if ((f >> 2) & 1u) topk_insert(tj, ti, &tcnt, k, J, idx);
            if (flag_dump) flag_dump[t] = f;
            if (J_dump) J_dump[t] = J;
            if (pred_dump)
                for (int i = 0; i < N; i++) {
                    pred_dump[((size_t)t * N + i) * 2 + 0] = lat[i];
                    pred_dump[((size_t)t * N + i) * 2 + 1] = thr[i];
                }
        }
#pragma omp critical
        {
            n_vram += lv;
            n_feas += lf;
            n_inexact += lx;
            for (int b = 0; b < 4; b++) near[b] += ln[b];
            for (int q = 0; q < tcnt; q++) topk_insert(gJ, gI, &gcnt, k, tj[q], ti[q]);
        }
        free(scr);
    }
    out->n_eval = (uint64_t)n;
    out->n_vram = n_vram;
    out->n_feas = n_feas;
    out->n_inexact_agg = n_inexact;
    for (int b = 0; b < 4; b++) out->n_near[b] = near[b];
    out->n_top = gcnt;
    for (int q = 0; q < ORC_MAX_TOPK; q++) {
        out->top_idx[q] = q < gcnt ? gI[q] : UINT64_MAX;
        out->top_J[q] = q < gcnt ? gJ[q] : -INFINITY;
    }
    free(w64);
    return 0;
}

/* Canonical evaluation of a list of configurations (sampled parity at sizes
 * too large for brute force).  lat/thr: [n][N]; J, flags: [n]. */
int orc_eval_list(const orc_instance *in, const uint64_t *idx, int64_t n, const float *sla,
                  const float *omega, int nthreads, double *lat, double *thr, double *J,
                  uint32_t *flags)
{
    const int N = in->n_models;
    double *w64 = orc_weights_f64(in);
    if (!w64) return -1;
    if (nthreads < 1) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads)
    {
        double *scr = (double *)malloc(sizeof(double) * orc_scratch_doubles(in));
#pragma omp for schedule(static)
        for (int64_t t = 0; t < n; t++)
            orc_eval_w(in, w64, idx[t], sla, omega, lat + t * N, thr + t * N, J + t, flags + t, scr);
        free(scr);
    }
    free(w64);
    return 0;
}

/* Ascending list of the VRAM-feasible indices (the constructed feasible space
 * of Section II).  Returns the count; writes at most cap entries. */
uint64_t orc_vram_feasible(const orc_instance *in, uint32_t *list, uint64_t cap)
{
    uint64_t size = orc_space_size(in), cnt = 0;
    int32_t d[ORC_MAX_MODELS];
    float a[ORC_MAX_AGG];
    for (uint64_t idx = 0; idx < size; idx++) {
        orc_decode(in, idx, d);
        orc_aggregate(in, d, a);
        if ((double)a[in->vram_slot] <= (double)in->vram_cap) {
            if (cnt < cap) list[cnt] = (uint32_t)idx;
            cnt++;
        }
    }
    return cnt;
}

double orc_bf16_round(double x) { return bf16_round(x); }
