/*
 * mf.h: C ABI of the MeanField joint-configuration search for MI355X (gfx950).
 *
 * The method (Ennouri and Ha, "MeanField Surrogate Modeling for Scalable
 * Runtime Scheduling of Concurrent Heterogeneous AI Inference on Shared GPUs"):
 * N models share one GPU; model i runs one option from its discrete set
 * Lambda_i (Section II); a joint configuration picks one option per model
 * (Eq. 1).  A per-model surrogate g_i predicts the model's performance from its
 * own option and an aggregate GPU state (Section III-B, Eq. 6); the scheduler
 * takes the argmax of a utility J over the joint space (Section II, decision
 * rule before Eq. 3) subject to a VRAM cap and per-model service bounds (Eq. 4);
 * infeasible candidates score -inf and are never chosen.
 *
 * This library evaluates that decision step over a whole index range of the
 * joint space (exhaustive surrogate search, Section IV-C) or over a genetic
 * algorithm's population (the GA scheduler of Section IV-C), on the GPU.
 *
 * Conventions for every entry point:
 *  - Every call returns mf_status.  Arguments are validated on the host before
 *    anything is launched; on an error nothing has been enqueued.  No call
 *    prints, throws or exits.
 *  - Pointers prefixed d_ are device memory (any allocation the HIP runtime
 *    accepts, e.g. torch tensors); h_ are host memory.  All are caller-owned
 *    and borrowed only for the duration of the call unless stated otherwise.
 *  - `stream` is a hipStream_t (0 = the null stream) passed as void*.
 *  - Calls that return results on the host (mf_search, mf_ga_run) synchronise
 *    the stream before returning.  Others only enqueue work.
 *  - A problem may be used from several streams at once provided each call
 *    gets its own workspace.  Calls sharing one workspace must not overlap.
 *
 * Definitions (all indices 0-based):
 *  - Joint index: lexicographic order over (lambda_0, ..., lambda_{N-1}),
 *    model 0 most significant (the order of itertools.product).
 *  - Option table F: float [sum_i K_i][L] row-major; model i's K_i rows start
 *    at row sum_{j<i} K_j.
 *  - Aggregate state a (Eq. 2 recast per candidate): slot k is the fp32 sum,
 *    in model order 0..N-1, of column agg_cols[k] of every model's chosen row
 *    (each model's own row included).
 *  - Surrogate of model i (Eq. 6): z = [F row of lambda_i (L) | a (A)],
 *    h1 = relu(W1 z + b1), h2 = relu(W2 h1 + b2), (lat, thr) = out(W3 h2 + b3)
 *    with out the identity or, for MF_ACT_SIGMOID (the predictor's sigmoid
 *    output, Section III-B), s(y) = 1 / (1 + e^-y) on y clamped to
 *    [-700, 700].  Canonically e^x is this algorithm: k = rint(x * (1/ln 2)),
 *    r = fma(-k, ln2_hi, x) then r = fma(-k, ln2_lo, r) (ln2_hi = ln 2 to 24
 *    significant bits), e^r = the degree-13 Taylor polynomial by Horner with
 *    fma and coefficients 1/n! each rounded once, times 2^k.
 *  - Feasible: a[vram_slot] <= vram_cap and lat_i <= sla_i for every i
 *    (both inclusive, Eq. 4).  J = sum_i omega_i thr_i if feasible, else -inf.
 *  - Results are defined by canonical fp64 semantics: each dot product is one
 *    fused multiply-add chain in ascending input order starting from the bias,
 *    relu(x) = x > 0 ? x : +0, J is the fma chain over models in order.  In
 *    MF_BF16 mode W1, W2, W3 hold bfloat16 values and h1 is rounded to
 *    bfloat16 (nearest, ties to even) after the relu.  The GPU evaluates in
 *    fp32 (MFMA) and re-evaluates canonically every decision the fast path
 *    cannot prove (see mf_search), so counts, masks and top-k are exact.
 *  - Top-k order: J descending, then index ascending.
 */
#ifndef MF_H
#define MF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MF_OK = 0,
    MF_EINVAL = 1,        /* invalid argument (null pointer, bad size, non-finite value, ...) */
    MF_ENOMEM = 2,        /* workspace smaller than mf_workspace_size reports, or host allocation failed */
    MF_EDEVICE = 3,       /* a HIP runtime call or kernel launch failed */
    MF_EUNSUPPORTED = 4,  /* shape outside what the kernels are built for (see mf_desc) */
    MF_EOVERFLOW = 5,     /* prod K_i does not fit in 64 bits, or a range bound exceeds |Lambda| */
    MF_EINTERNAL = 6,     /* a self-check failed (fast-path error bound violated); result unusable */
    MF_ESCRATCH = 7       /* mf_search_noalloc: the search needs more than MF_NOALLOC_SCRATCH_BYTES */
} mf_status;

typedef enum { MF_F32 = 0, MF_BF16 = 1 } mf_dtype;

typedef enum { MF_ACT_IDENTITY = 0, MF_ACT_SIGMOID = 1 } mf_activation;

#define MF_MAX_MODELS 16
#define MF_MAX_TOPK 64

typedef struct mf_problem mf_problem;   /* opaque */

#define MF_MAX_VARIANTS 4

/* Variant metadata of the full utility (Section II, Eq. 3): an option set is
 * variants x runtime parameters, and each variant v of model i carries the
 * throughput extremes observed for it (f_i is min-max scaled per variant), a
 * quality Q, and model i a reload cost c_i.  Host arrays, copied at creation.
 * Validation: 1 <= n_variants[i] <= MF_MAX_VARIANTS, 0 <= variant < n_variants,
 * fmin < fmax, all values finite, reload costs >= 0; else MF_EINVAL. */
typedef struct {
    const int32_t *h_variant;      /* [sum K_i] variant of each option row */
    const int32_t *h_n_variants;   /* [N] */
    const float *h_fmin;           /* [N][MF_MAX_VARIANTS] */
    const float *h_fmax;           /* [N][MF_MAX_VARIANTS] */
    const float *h_quality;        /* [N][MF_MAX_VARIANTS] */
    const float *h_reload_cost;    /* [N] */
} mf_variants;

/* Problem shape.  Creation accepts 1 <= n_models <= 16, 1 <= n_options[i] <=
 * 255, n_local >= 1, 1 <= n_agg <= 16, n_local + n_agg <= 64, hidden sizes up
 * to 256.  The derived-state search (mf_search without MF_FIXED_STATE) needs
 * n_agg in {2,4,6,8} and hidden1 == hidden2 in {32, 64} for MF_F32, in
 * {64, 128, 256} for MF_BF16; the GA needs (hidden1, hidden2) in {(32, 32),
 * (64, 32), (64, 64)} with fixed input widths (mf_ga_run); the fixed-state
 * and static searches take any created shape.  Other combinations return
 * MF_EUNSUPPORTED from the call that needs them.  Trained predictors with
 * batch normalisation fold it into the preceding layer's weights and bias
 * before creation (an affine map at inference). */
typedef struct {
    int32_t n_models;           /* N */
    int32_t n_local;            /* L: local features per option row */
    int32_t n_agg;              /* A: aggregate slots */
    int32_t hidden1, hidden2;   /* H1, H2; the output layer has 2 units: [0] latency, [1] throughput */
    const int32_t *h_n_options; /* host [N] */
    const int32_t *h_agg_cols;  /* host [A], each in [0, L) */
    int32_t vram_slot;          /* aggregate slot compared with vram_cap, in [0, A) */
    float vram_cap;             /* finite */
    mf_dtype dtype;
    const mf_variants *variants; /* NULL: only the linear objective is available */
    int32_t output_act;          /* mf_activation of both surrogate outputs (zero: identity) */
} mf_desc;

/* Bytes of caller-owned device memory a problem of this description needs
 * for its tables (the option sets Lambda_i = V_i x P_i of Section II as
 * option rows, one surrogate g_i per model, Section III-B / Eq. 6, and the
 * fast paths' images of both).  A function of the description's shape only:
 * the pointers to option counts and aggregate columns are read, no weights.
 * Errors: MF_EINVAL / MF_EOVERFLOW as mf_problem_create. */
mf_status mf_problem_bytes(const mf_desc *desc, size_t *bytes);

/* Create a problem: the option sets Lambda_i (Section II), one row of L local
 * features per option, and the per-model surrogates g_i of Eq. 6 (Section
 * III-B).  d_features: float [sum K_i][L].  d_weights: float [N][S] with
 * S = H1*(L+A) + H1 + H2*H1 + H2 + 2*H2 + 2, per model packed as W1[H1][L+A],
 * b1[H1], W2[H2][H1], b2[H2], W3[2][H2], b3[2] (row-major).  Both are read on
 * `stream` (device or host memory) and copied: the caller may free them after
 * the call returns.  d_tables: caller-owned device memory of at least
 * mf_problem_bytes(desc) bytes, 256-byte aligned (else MF_ENOMEM / MF_EINVAL),
 * which the problem uses for all its tables; it must stay allocated and
 * unmodified until mf_problem_destroy.  The library allocates no device
 * memory.  Validates every value is finite (and bf16-representable for
 * MF_BF16 W*), derives the fast path's error bounds, and writes the tables
 * (per-option first-layer precompute included) on `stream`; returns after the
 * stream has finished that work. */
mf_status mf_problem_create(const mf_desc *desc, const float *d_features, const float *d_weights,
                            void *d_tables, size_t table_bytes, void *stream, mf_problem **out);
/* Releases the host state; d_tables is the caller's to free afterwards. */
void mf_problem_destroy(mf_problem *p);

/* |Lambda| = prod K_i, the size of the joint configuration space of Eq. 1. */
mf_status mf_space_size(const mf_problem *p, uint64_t *out);

/* Host helper: the options (lambda_0, ..., lambda_{N-1}) of joint index idx
 * (Eq. 1: lexicographic order, model 0 most significant) into digits[N];
 * MF_EINVAL when idx >= |Lambda|. */
mf_status mf_decode(const mf_problem *p, uint64_t idx, int32_t *h_digits);

/* ---------------------------------------------------------------- search */

#define MF_DUMP 1u   /* write d_mask and d_pred for every index of [lo, hi) */
#define MF_FIXED_STATE 2u  /* hold the surrogates' aggregate input at `state` (see mf_search_args) */
#define MF_MAX_AGG 16

typedef enum {
    MF_OBJ_LINEAR = 0,  /* J = sum_i omega_i thr_i (Section II with unit quality) */
    MF_OBJ_EQ3 = 1      /* the full utility of Eq. 3 with the throughput floor (needs mf_desc.variants) */
} mf_objective_kind;

/* Objective of a search.  MF_OBJ_EQ3 (Section II, Eq. 3 and the constraint
 * after it), with v the variant of model i's option:
 *   f_i = (thr_i - fmin_{i,v}) / (fmax_{i,v} - fmin_{i,v})
 *   J   = sum_i omega_i Q_{i,v} f_i - alpha sum_i eta_i c_i
 *         - beta sum_i max(0, tau_i + delta - f_i)^2,
 *   eta_i = 1 iff prev_variant[i] >= 0 and v != prev_variant[i];
 * feasible additionally requires f_i >= tau_i (tau_i = -inf: no floor).
 * Canonical evaluation per model, in fp64 and in this order: Rg = fmax - fmin,
 * f = (thr - fmin) / Rg, q = Q f, J = fma(omega, q, J), J = J - alpha c (if
 * eta), d = (tau + delta) - f, J = J - beta (d d) (if d > 0).  The latency
 * bounds d_sla still apply (pass +inf to drop them).  Validation: alpha, beta,
 * delta finite, beta >= 0; tau not NaN or +inf; -1 <= prev_variant[i] < n_variants[i]. */
typedef struct {
    int32_t kind;                           /* mf_objective_kind */
    float alpha, beta, delta;
    float tau[MF_MAX_MODELS];
    int32_t prev_variant[MF_MAX_MODELS];
} mf_objective;

typedef struct {
    uint64_t lo, hi;           /* half-open index range, lo <= hi <= |Lambda| */
    int32_t top_k;             /* 1..64 */
    uint32_t flags;            /* MF_DUMP | MF_FIXED_STATE */
    const float *d_sla;        /* device [N] latency bound per model (+inf: none) */
    const float *d_omega;      /* device [N] objective weight per model, finite */
    /* MF_DUMP outputs (device, hi - lo <= 2^31 entries):
     *   d_mask[t]: bit0 VRAM ok, bit1 every service constraint met (latency
     *              bounds; throughput floors under MF_OBJ_EQ3), bit2 feasible,
     *              bit3 the fast path left a service decision to the
     *              canonical re-evaluation;
     *   d_pred[(t*N + i)*2 + {0,1}]: fast-path fp32 (lat, thr) of model i
     *              (MF_FIXED_STATE: the canonical values rounded to fp32). */
    uint8_t *d_mask;
    float *d_pred;
    mf_objective objective;    /* zero-initialised: MF_OBJ_LINEAR */
    /* MF_FIXED_STATE (Section III-B: the aggregate GPU state is observed by
     * the runtime monitor and held fixed during the search): every surrogate
     * takes state[0..A) (original slot order, finite) as its aggregate input
     * instead of the candidate's own aggregate, so model i's prediction
     * depends on its option only; the VRAM constraint still sums the
     * candidate's options.  The search then runs the surrogates once per
     * option row (canonical semantics) and scans the joint space over those
     * tables, exactly: any created shape is supported (no fast-path shape
     * limits), d_pred receives the canonical (lat, thr) rounded to fp32, mask
     * bit3 and n_flagged / n_topk_collect / n_splits stay 0. */
    float state[MF_MAX_AGG];
    /* Upper bound on the entries of the certification list (configurations
     * whose service decision the fast path leaves to the canonical
     * re-evaluation); 0 keeps the default (1/64 of the range, at least 2^20,
     * at most 2^26).  A smaller list shrinks the workspace; a range that fills
     * it is split in halves and searched again (n_splits). */
    uint32_t worklist_cap;
} mf_search_args;

typedef struct {
    uint64_t n_eval;           /* hi - lo */
    uint64_t n_vram;           /* VRAM-feasible configurations */
    uint64_t n_feas;           /* feasible (VRAM and every service constraint) */
    uint64_t n_flagged;        /* configurations re-evaluated canonically for a latency decision */
    uint64_t n_topk_collect;   /* candidates gathered by the top-k fallback pass (0 if none ran) */
    int32_t n_top;             /* min(top_k, n_feas) */
    int32_t n_splits;          /* range splits forced by a full certification list */
    uint64_t top_idx[MF_MAX_TOPK];  /* joint indices; UINT64_MAX past n_top */
    double top_J[MF_MAX_TOPK];      /* canonical J; -inf past n_top */
    float main_kernel_ms;      /* HIP-event time of the fast search kernel(s) on `stream` */
    float pad;
} mf_result;

/* Bytes of device workspace mf_search needs for these arguments. */
mf_status mf_workspace_size(const mf_problem *p, const mf_search_args *args, size_t *bytes);

/* Exhaustive surrogate search over [lo, hi) (Section IV-C): counts, and the
 * exact top-k under canonical semantics.  d_ws: device workspace of at least
 * mf_workspace_size bytes (contents need not be initialised; 256-byte
 * aligned).  Blocking: returns after the result is on the host in *h_out.
 * Empty feasible set: MF_OK with n_top = 0. */
mf_status mf_search(mf_problem *p, const mf_search_args *args, void *d_ws, size_t ws_bytes,
                    void *stream, mf_result *h_out);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): mf_search
 * with its workspace taken from a fixed device scratch array that the library
 * holds, one copy per GPU, until the process ends.  Same arguments, results
 * and blocking behaviour as mf_search; the call allocates nothing (no
 * hipMalloc, no library allocation; timing uses events created with the
 * problem, and runs untimed, main_kernel_ms = 0, when another call holds
 * them).  MF_ESCRATCH when mf_workspace_size(args) exceeds
 * MF_NOALLOC_SCRATCH_BYTES: lower args->worklist_cap or search a shorter
 * range.  The current device must be the problem's (else MF_EINVAL).  Every
 * call on one GPU uses that GPU's single scratch array: calls that overlap on
 * one GPU (other threads, other streams) race and give wrong results;
 * serialise them.  The scratch keeps the last call's contents; each call
 * initialises what it reads. */
#define MF_NOALLOC_SCRATCH_BYTES (128u << 20)
mf_status mf_search_noalloc(mf_problem *p, const mf_search_args *args, void *stream, mf_result *h_out);

/* ------------------------------------------------- static (multi-step) search */

#define MF_MAX_STEPS 32

/* One configuration held over T decision steps: the static schedulers of
 * Section IV-C (Table II; StaticFull picks it with access to the whole
 * space).  Step t evaluates every surrogate at the observed state
 * h_state[t] (Section III-B, as MF_FIXED_STATE), with the step's latency
 * bounds d_sla[t] and weights d_omega[t]; the previous deployment is
 * objective.prev_variant at step 0 and the configuration itself afterwards
 * (no reload after step 0).  J_t is the step's canonical utility (as
 * mf_search computes it) and S = ((J_0 + J_1) + J_2) + ... in step order,
 * fp64.  A configuration is feasible when its VRAM sum meets the cap and
 * every step's latency bounds (and floors under MF_OBJ_EQ3) hold. */
typedef struct {
    uint64_t lo, hi;           /* half-open index range (search) */
    int32_t top_k;             /* 1..64 (search) */
    int32_t n_steps;           /* T, 1..MF_MAX_STEPS */
    const float *d_sla;        /* device [T][N] */
    const float *d_omega;      /* device [T][N], finite */
    const float *h_state;      /* host [T][A] observed aggregate per step, finite */
    mf_objective objective;    /* MF_OBJ_LINEAR or MF_OBJ_EQ3 (shared by the steps) */
    uint8_t *d_mask;           /* optional device [hi - lo] (search, hi - lo <= 2^31): bit0 VRAM ok,
                                  bit1 every step's service constraints met, bit2 feasible */
} mf_static_args;

/* Bytes of device workspace mf_search_static / mf_eval_static need. */
mf_status mf_static_workspace_size(const mf_problem *p, const mf_static_args *args, size_t *bytes);

/* argmax of S over the configurations of [lo, hi) feasible at every step;
 * counts (n_vram, n_feas) and the exact top-k by (S desc, index asc) in
 * h_out (top_J holds S).  Any created shape; T x sum K_i option rows must
 * fit in LDS (MF_EUNSUPPORTED otherwise).  Blocking. */
mf_status mf_search_static(mf_problem *p, const mf_static_args *args, void *d_ws, size_t ws_bytes,
                           void *stream, mf_result *h_out);

/* Per-step evaluation of an index list: d_J [n][T] the utility J_t (its
 * value also where a constraint fails), d_S [n] the step-order sum, d_flags
 * [n][T] (bit0 VRAM ok, bit1 the step's service constraints met).  Any
 * output may be NULL; lo, hi, top_k and d_mask are ignored.  With T = 1 and
 * objective.prev_variant set to the previous decision it evaluates one
 * step of a dynamic schedule.  Blocking. */
mf_status mf_eval_static(mf_problem *p, const mf_static_args *args, const uint64_t *d_idx, int64_t n,
                         double *d_J, double *d_S, uint32_t *d_flags, void *d_ws, size_t ws_bytes,
                         void *stream);

/* ------------------------------------------------------------ evaluation */

/* Fast-path predictions of an index list: (lat_i, thr_i) = g_i([x_i | a])
 * of Eq. 6 for every model of each joint configuration (aggregate derived
 * from the configuration, Section II), as the search kernel computes them
 * (fp32, or bf16 products with fp32 accumulation, on MFMA).  d_idx: device
 * uint64 [n], each < |Lambda|.  d_pred: device float [n][N][2] (lat, thr).
 * Enqueues only. */
mf_status mf_eval_fast(mf_problem *p, const uint64_t *d_idx, int64_t n, float *d_pred, void *stream);

/* Canonical fp64 evaluation of an index list (the semantics results are
 * defined by): the predictions of Eq. 6, the constraints of Eq. 4 and the
 * objective J of Section II for each joint configuration.  d_pred: device double [n][N][2]; d_J: device double [n]
 * (-inf when infeasible); d_flags: device uint32 [n] (bit0 VRAM ok, bit1 all
 * latency bounds met, bit2 feasible, bit 8+i model i misses its bound).  Any
 * output may be NULL.  Enqueues only. */
mf_status mf_eval_canonical(mf_problem *p, const uint64_t *d_idx, int64_t n, const float *d_sla,
                            const float *d_omega, double *d_pred, double *d_J, uint32_t *d_flags,
                            void *stream);

/* -------------------------------------------------------------------- GA */

/* Genetic-algorithm scheduler (Section IV-C) over S independent scenarios,
 * each with its own latency bounds and objective weights.  Fitness is the
 * canonical J of each individual (the same decode, aggregate, surrogate, mask
 * and score steps as the search, including the objective and the fixed
 * observed state when given).  Random draws come from Philox4x64-10
 * (Salmon et al., SC'11) keyed by `seed`; see mf_ga.hip for the counter
 * layout and operator order. */
typedef struct {
    int32_t n_scen;            /* S >= 1 */
    int32_t pop;               /* population, even, 4..4096 */
    int32_t gens;              /* offspring generations (>= 0); (gens+1)*pop evaluations per scenario */
    int32_t tourn_k;           /* tournament size 1..8 (with replacement) */
    float p_cx;                /* crossover probability per parent pair */
    float p_swap;              /* per-gene swap probability inside a crossover */
    float p_mut;               /* per-gene mutation probability */
    float pad;
    uint64_t seed;
    const float *d_sla;        /* device [S][N] */
    const float *d_omega;      /* device [S][N] */
    uint32_t flags;            /* MF_FIXED_STATE: the surrogates see state[] (as in mf_search) */
    float state[MF_MAX_AGG];   /* MF_FIXED_STATE: observed aggregate, original slot order, finite */
    mf_objective objective;    /* zero-initialised: MF_OBJ_LINEAR; MF_OBJ_EQ3 as in mf_search */
    /* Optional host output (NULL: none): the individuals of the run whose
     * fitness ran the surrogates.  Large populations (S x pop > 8192, shapes
     * with the one-lane fitness kernel) over joint spaces small enough to
     * tabulate (|Lambda| (16 N + 4) bytes <= 256 MiB) keep a memo of each
     * evaluated index's canonical predictions in the workspace for the rest of
     * the run; later generations read it (the values, and so the trajectory,
     * are the same).  Otherwise every individual counts. */
    uint64_t *h_forwards;
} mf_ga_args;

mf_status mf_ga_workspace_size(const mf_problem *p, const mf_ga_args *args, size_t *bytes);

/* Runs the GA.  h_best_idx / h_best_J: host [S], the best individual ever
 * evaluated per scenario (J desc, index asc); UINT64_MAX / -inf if none was
 * feasible.  d_final_pop (optional, device uint64 [S][pop]): the last
 * population's joint indices, all UINT64_MAX when no configuration meets the
 * VRAM cap.  Blocking (one synchronisation, at the end). */
mf_status mf_ga_run(mf_problem *p, const mf_ga_args *args, void *d_ws, size_t ws_bytes,
                    void *stream, uint64_t *h_best_idx, double *h_best_J, uint64_t *d_final_pop);

/* Human-readable status name. */
const char *mf_status_string(mf_status s);

#ifdef __cplusplus
}
#endif

#endif /* MF_H */
