/* Types shared by the CPU oracle's C files (test infrastructure only). */
#ifndef MF_ORACLE_H
#define MF_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#define ORC_MAX_MODELS 16
#define ORC_MAX_TOPK 64
#define ORC_MAX_AGG 16
#define ORC_MAX_VARIANTS 4

/* The full utility of Section II (Eq. 3) with the throughput floor of the
 * constraint after it; NULL in orc_instance selects J = sum_i omega_i thr_i
 * with the latency bounds as the only service constraint. */
typedef struct {
    const int32_t *variant;       /* [sum K] variant of each option row */
    const float *fmin, *fmax;     /* [N][ORC_MAX_VARIANTS] per-variant throughput extremes */
    const float *quality;         /* [N][ORC_MAX_VARIANTS] Q of each variant */
    const float *reload_cost;     /* [N] c_i^rel */
    const int32_t *prev_variant;  /* [N] variant deployed at the previous step, -1 for none */
    const float *tau;             /* [N] floor on the normalised throughput (-inf: none) */
    float alpha, beta, delta;
} orc_objective;

typedef struct {
    int32_t n_models, n_local, n_agg, hidden1, hidden2, bf16;
    const int32_t *n_options;   /* [N] */
    const float *features;      /* [sum K][L] row-major, model i at offset sum_{j<i} K_j */
    const int32_t *agg_cols;    /* [A] */
    int32_t vram_slot;
    float vram_cap;
    const float *weights;       /* [N][stride]: W1[h1][L+A] b1[h1] W2[h2][h1] b2[h2] W3[2][h2] b3[2] */
    const orc_objective *obj;   /* NULL: linear objective */
    const float *fixed_state;   /* [A] observed aggregate state fed to every surrogate (Section III-B:
                                   held fixed during the search); NULL: derived from each candidate */
    int32_t raw_J;              /* nonzero: J is the utility value also where a constraint fails
                                   (the flags still say which); for evaluating decisions that break
                                   a bound, as a random scheduler's do (Section IV-C, Table II) */
    int32_t sigmoid;            /* nonzero: both surrogate outputs pass a sigmoid (the predictor's
                                   output layer, Section III-B); zero: identity output */
} orc_instance;

double orc_exp(double x);
double orc_sigmoid(double y);

typedef struct {
    uint64_t n_eval, n_vram, n_feas;
    uint64_t n_inexact_agg;     /* configs whose fp32 aggregate differs from fp64 (expected 0) */
    uint64_t n_near[4];         /* (config, model) pairs with |lat - sla| <= {1e-5,1e-4,1e-3,2e-2} */
    int32_t n_top;
    int32_t pad;
    uint64_t top_idx[ORC_MAX_TOPK];
    double top_J[ORC_MAX_TOPK];
} orc_result;

uint64_t orc_space_size(const orc_instance *in);
void orc_decode(const orc_instance *in, uint64_t idx, int32_t *digits);
uint64_t orc_encode(const orc_instance *in, const int32_t *digits);
int orc_aggregate(const orc_instance *in, const int32_t *digits, float *a);
double *orc_weights_f64(const orc_instance *in);
size_t orc_scratch_doubles(const orc_instance *in);
void orc_eval_w(const orc_instance *in, const double *w64, uint64_t idx, const float *sla, const float *omega,
                double *lat, double *thr, double *J, uint32_t *flags, double *scratch);
uint64_t orc_vram_feasible(const orc_instance *in, uint32_t *list, uint64_t cap);

#endif
