"""Seeded synthetic scheduling instances shaped like the paper's workloads.

The paper (Section II) schedules N co-running inference models on one GPU.
Model i exposes a discrete option set Lambda_i = V_i x P_i (variants x runtime
parameters); the LLM family and the vision family are the two model types.
Its surrogate (Section III-B, Eq. 6) is one small MLP per model fed the model's
local configuration and the aggregate GPU state.  The paper's profiling tables
and trained weights are not published, so every table here is drawn from a
seeded PCG64 stream with the shapes the paper describes.

This module draws inputs only.  It holds no step of the method (no decode, no
aggregate, no surrogate evaluation, no masking or scoring): both the HIP path
and the CPU oracle receive the arrays it returns.

Feature columns of an option row (L >= 8):
  0  LLM one-hot          (constant per model: a model is one family)
  1  vision one-hot
  2  log2 batch           integer in {0..5}
  3  SM share             U[0.1, 1]
  4  VRAM (GB)            U[1, 40]
  5  bandwidth demand     U[0.05, 0.6]
  6+ noise                U[0, 1]
Continuous columns are quantised to multiples of 2**-14 by default, so every
aggregate sum of at most 16 rows is exact in fp32 whatever the summation
order; make_instance(..., quantise=False) keeps them off the grid.

Aggregate slots (each the sum over all N models of one option column):
  A=2: [sum SM, sum VRAM]
  A=4: [sum SM, sum VRAM, sum BW, #LLM]
  A=6: + [#vision, sum log2 batch]
  A=8: + [sum noise6, sum noise7]

Weights are N(0, 1/fan_in), biases 0, and input standardisation (per-column
mean and SD of the local features; mean and SD of each aggregate slot under a
uniform choice per model) is folded into the first layer, as a trained
surrogate with standardised inputs would carry it.
"""
from __future__ import annotations

from dataclasses import dataclass, field
import numpy as np

GRID = 2.0 ** -14
COL_LLM, COL_VIS, COL_LOG2B, COL_SM, COL_VRAM, COL_BW = 0, 1, 2, 3, 4, 5
AGG_COLS = {2: [COL_SM, COL_VRAM],
            4: [COL_SM, COL_VRAM, COL_BW, COL_LLM],
            6: [COL_SM, COL_VRAM, COL_BW, COL_LLM, COL_VIS, COL_LOG2B],
            8: [COL_SM, COL_VRAM, COL_BW, COL_LLM, COL_VIS, COL_LOG2B, 6, 7]}
VRAM_SLOT = 1
N_OUT = 2                       # [0] latency, [1] throughput
Z75 = 0.6744897501960817        # standard normal 75th percentile


def model_stride(n_in: int, h1: int, h2: int) -> int:
    """Floats per model in the packed weight block:
    W1[h1][n_in], b1[h1], W2[h2][h1], b2[h2], W3[2][h2], b3[2]."""
    return h1 * n_in + h1 + h2 * h1 + h2 + N_OUT * h2 + N_OUT


def unpack_model(weights_row: np.ndarray, n_in: int, h1: int, h2: int):
    """Split one model's packed weight row into (W1, b1, W2, b2, W3, b3) views."""
    o = 0
    out = []
    for shape in ((h1, n_in), (h1,), (h2, h1), (h2,), (N_OUT, h2), (N_OUT,)):
        size = int(np.prod(shape))
        out.append(weights_row[o:o + size].reshape(shape))
        o += size
    return tuple(out)


def _quantise(v: np.ndarray) -> np.ndarray:
    return np.round(v / GRID) * GRID


def _to_bf16_values(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (via fp32, ties to even); return fp32."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000
    return b.astype(np.uint32).view(np.float32)


@dataclass
class Instance:
    name: str
    n_options: np.ndarray          # int32 [N]
    model_type: np.ndarray         # int32 [N], 0 = LLM, 1 = vision
    n_local: int
    n_agg: int
    hidden1: int
    hidden2: int
    features: np.ndarray           # float32 [sum K][L]
    agg_cols: np.ndarray           # int32 [A]
    vram_slot: int
    vram_cap: float                # fp32 value
    weights: np.ndarray            # float32 [N][model_stride]
    sla: np.ndarray                # float32 [N] latency bound per model
    omega: np.ndarray              # float32 [N] objective weight per model
    dtype: str = "f32"             # "f32" or "bf16" (W1, W2, W3 hold bf16 values)
    top_k: int = 1
    seed: int = 0
    extra: dict = field(default_factory=dict)
    act: str = "identity"          # output activation: "identity" or "sigmoid" (the paper's predictor)

    @property
    def n_models(self) -> int:
        return int(self.n_options.shape[0])

    @property
    def n_in(self) -> int:
        return self.n_local + self.n_agg

    @property
    def space_size(self) -> int:
        return int(np.prod([int(k) for k in self.n_options], dtype=object))

    @property
    def option_offsets(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.n_options)[:-1]]).astype(np.int64)

    def model_weights(self, i: int):
        return unpack_model(self.weights[i], self.n_in, self.hidden1, self.hidden2)


def make_instance(n_options, n_local=8, n_agg=4, hidden1=32, hidden2=32, *,
                  seed=0, dtype="f32", vram_cap=None, vram_quantile=None,
                  sla_range=(0.5, 2.0), top_k=1, types=None,
                  symmetric=False, name="custom", act="identity", quantise=True) -> Instance:
    """Draw one instance.

    n_options: option count per model.  types: per-model family (0 LLM, 1
    vision); default: the first ceil(N/2) models are LLMs, as in the paper's
    N=2 (one LLM, one YOLO) and N=5 (three LLMs, two YOLO) mixes.
    vram_cap: fixed cap in GB; vram_quantile: cap set at that quantile of the
    normal approximation to the joint VRAM sum (a uniform choice per model).
    symmetric: copy model 0's option table and weights to every model (all
    options counts must agree).  act: the surrogates' output activation
    ("sigmoid": outputs in (0, 1), so latency bounds belong in (0, 1)).
    quantise: put the continuous feature columns on the 2^-14 grid (default;
    every aggregate sum is then exact in fp32 whatever the order); False keeps
    the drawn values rounded to fp32 only, as real profiling tables would
    come, so the aggregate's fp32 sums round.
    """
    if act not in ("identity", "sigmoid"):
        raise ValueError(f"unknown output activation {act!r}")
    n_options = np.asarray(n_options, dtype=np.int32)
    N = int(n_options.shape[0])
    if n_local < 8:
        raise ValueError("n_local must be >= 8 (the column layout needs 8)")
    if n_agg not in AGG_COLS:
        raise ValueError(f"n_agg must be one of {sorted(AGG_COLS)}")
    if types is None:
        types = [0 if i < (N + 1) // 2 else 1 for i in range(N)]
    types = np.asarray(types, dtype=np.int32)
    rng = np.random.Generator(np.random.PCG64(seed))
    L, A = n_local, n_agg
    n_in = L + A
    q = _quantise if quantise else (lambda v: v.astype(np.float32).astype(np.float64))

    # --- option tables ---
    rows = []
    for i in range(N):
        K = int(n_options[i])
        f = np.zeros((K, L), dtype=np.float64)
        f[:, COL_LLM] = 1.0 if types[i] == 0 else 0.0
        f[:, COL_VIS] = 1.0 if types[i] == 1 else 0.0
        f[:, COL_LOG2B] = rng.integers(0, 6, K)
        f[:, COL_SM] = q(rng.uniform(0.1, 1.0, K))
        f[:, COL_VRAM] = q(rng.uniform(1.0, 40.0, K))
        f[:, COL_BW] = q(rng.uniform(0.05, 0.6, K))
        f[:, 6:] = q(rng.uniform(0.0, 1.0, (K, L - 6)))
        rows.append(f)
    if symmetric:
        if len(set(int(k) for k in n_options)) != 1:
            raise ValueError("symmetric instances need equal option counts")
        rows = [rows[0].copy() for _ in range(N)]
        types[:] = types[0]
    feats64 = np.concatenate(rows, axis=0)
    agg_cols = np.asarray(AGG_COLS[A], dtype=np.int32)

    # --- standardisation statistics (generator-side weight synthesis) ---
    mu_loc = feats64.mean(axis=0)
    sd_loc = feats64.std(axis=0)
    mu_agg = np.zeros(A)
    var_agg = np.zeros(A)
    for i in range(N):
        for j, c in enumerate(agg_cols):
            mu_agg[j] += rows[i][:, c].mean()
            var_agg[j] += rows[i][:, c].var()
    sd_agg = np.sqrt(var_agg)
    mu = np.concatenate([mu_loc, mu_agg])
    sd = np.concatenate([sd_loc, sd_agg])
    sd[sd == 0.0] = 1.0

    # --- surrogate weights ---
    stride = model_stride(n_in, hidden1, hidden2)
    weights = np.zeros((N, stride), dtype=np.float32)
    for i in range(N):
        W1 = rng.standard_normal((hidden1, n_in)) / np.sqrt(n_in)
        W2 = rng.standard_normal((hidden2, hidden1)) / np.sqrt(hidden1)
        W3 = rng.standard_normal((N_OUT, hidden2)) / np.sqrt(hidden2)
        W1f = W1 / sd[None, :]
        b1f = -(W1f @ mu)
        if dtype == "bf16":
            W1q, W2q, W3q = (_to_bf16_values(w) for w in (W1f, W2, W3))
        elif dtype == "f32":
            W1q, W2q, W3q = (w.astype(np.float32) for w in (W1f, W2, W3))
        else:
            raise ValueError("dtype must be 'f32' or 'bf16'")
        parts = [W1q.ravel(), b1f.astype(np.float32), W2q.ravel(),
                 np.zeros(hidden2, np.float32), W3q.ravel(), np.zeros(N_OUT, np.float32)]
        weights[i] = np.concatenate(parts)
    if symmetric:
        weights[1:] = weights[0]

    # --- constraint parameters ---
    lo, hi = sla_range
    sla = rng.uniform(lo, hi, N).astype(np.float32)
    if symmetric:
        sla[:] = sla[0]
    omega = np.ones(N, dtype=np.float32)
    if vram_cap is None:
        if vram_quantile is None:
            raise ValueError("give vram_cap or vram_quantile")
        m = sum(r[:, COL_VRAM].mean() for r in rows)
        v = sum(r[:, COL_VRAM].var() for r in rows)
        z = {0.75: Z75}.get(vram_quantile)
        if z is None:
            from statistics import NormalDist
            z = NormalDist().inv_cdf(vram_quantile)
        vram_cap = m + z * np.sqrt(v)
    return Instance(name=name, n_options=n_options, model_type=types, n_local=L,
                    n_agg=A, hidden1=hidden1, hidden2=hidden2,
                    features=feats64.astype(np.float32), agg_cols=agg_cols,
                    vram_slot=VRAM_SLOT, vram_cap=float(np.float32(vram_cap)),
                    weights=weights, sla=sla, omega=omega, dtype=dtype,
                    top_k=top_k, seed=seed, act=act)


# ---------------------------------------------------------------------------
# The five workloads (sizes from the scheduling study: N=2..8 models)
# ---------------------------------------------------------------------------

def cfg0(seed=0) -> Instance:
    """N=2, 6 options each (36 joint configs), 12->32->32->2 fp32, VRAM cap
    80 GB, argmax."""
    return make_instance([6, 6], 8, 4, 32, 32, seed=seed, vram_cap=80.0,
                         top_k=1, name="n2_k6x6_h32")


def cfg1(seed=0) -> Instance:
    """N=5, options (12,12,9,9,9) = 104,976 joint configs, same MLP; VRAM cap
    at the 75th percentile of the joint VRAM sum (about 78k feasible); top-16."""
    return make_instance([12, 12, 9, 9, 9], 8, 4, 32, 32, seed=seed,
                         vram_quantile=0.75, top_k=16, name="n5_k12x12x9x9x9_h32")


def cfg2(seed=0) -> Instance:
    """N=6, 24 options each (191,102,976 joint configs), L=16, A=6,
    22->64->64->2 fp32, VRAM cap 200 GB, argmax + feasible count."""
    return make_instance([24] * 6, 16, 6, 64, 64, seed=seed, vram_cap=200.0,
                         top_k=1, name="n6_k24_h64")


def paper_predictor(seed=0) -> Instance:
    """The N=5 option sets with the paper's predictor architecture (Section
    III-B): hidden layers 64 and 32, sigmoid outputs (batch norm folded,
    dropout the identity at inference).  The latency bounds sit at 0.75; the
    scheduling protocol replaces them per step."""
    return make_instance([12, 12, 9, 9, 9], 8, 4, 64, 32, seed=seed, vram_quantile=0.75, sla_range=(0.75, 0.75),
                         top_k=16, name="n5_paper_64_32_sigmoid", act="sigmoid")


def cfg4(seed=0) -> Instance:
    """N=8, 16 options each (2**32 joint configs), L=32, A=8,
    40->256->256->2 with bf16 weights, VRAM cap 288 GB, top-64."""
    return make_instance([16] * 8, 32, 8, 256, 256, seed=seed, vram_cap=288.0,
                         dtype="bf16", top_k=64, name="n8_k16_h256_bf16")


def _slot_stats(inst: Instance):
    """Mean and SD of each aggregate slot under a uniform choice per model,
    from the option tables alone."""
    offs = np.concatenate([[0], np.cumsum(inst.n_options)])
    mu = np.zeros(inst.n_agg)
    var = np.zeros(inst.n_agg)
    for k, c in enumerate(inst.agg_cols):
        for i in range(inst.n_models):
            col = inst.features[offs[i]:offs[i + 1], c].astype(np.float64)
            mu[k] += col.mean()
            var[k] += col.var()
    return mu, np.sqrt(var)


def make_state(inst: Instance, seed: int = 0, spread: float = 0.5) -> np.ndarray:
    """An observed aggregate state (what the runtime monitor reports,
    Section II), float32 [A]: each slot drawn around its mean under a uniform
    choice per model, `spread` standard deviations wide, on the 2^-14 grid.
    The statistics come from the option tables alone."""
    rng = np.random.Generator(np.random.PCG64(seed * 104729 + 3))
    mu, sd = _slot_stats(inst)
    st = np.array([mu[k] + spread * sd[k] * rng.standard_normal() for k in range(inst.n_agg)])
    return _quantise(st).astype(np.float32)


@dataclass
class Scenarios:
    """Dynamic scenarios of the scheduling protocol (Section IV-C, Table II):
    per scenario s and decision step t the observed aggregate state, the
    latency bounds and the objective weights."""
    states: np.ndarray           # float32 [S][T][A]
    sla: np.ndarray              # float32 [S][T][N]
    omega: np.ndarray            # float32 [S][T][N]
    elevated: np.ndarray         # int32 [S]: the model whose weight a scenario raises


def make_scenarios(inst: Instance, n_scen: int = 8, n_steps: int = 12, seed: int = 0, rho: float = 0.8,
                   walk: float = 0.3, elevate: float = 2.0, latency_bounds: bool = False) -> Scenarios:
    """Seeded dynamic scenarios.  The observed state follows an AR(1) walk per
    slot toward the slot mean (start mean + 0.5 SD z, then mean + rho (x -
    mean) + walk SD z), on the 2^-14 grid; one model per scenario has its
    weight raised to `elevate` over a window of steps (the others 1: Section
    II sets omega_i = 1 unless a scenario elevates one).  The service
    constraint is the throughput floor of Eq. 3, so the latency bounds are
    +inf unless latency_bounds (then the instance's bounds at every step)."""
    N, A, T = inst.n_models, inst.n_agg, n_steps
    mu, sd = _slot_stats(inst)
    states = np.zeros((n_scen, T, A), np.float32)
    sla = np.full((n_scen, T, N), np.inf, np.float32)
    omega = np.ones((n_scen, T, N), np.float32)
    elevated = np.zeros(n_scen, np.int32)
    for s in range(n_scen):
        rng = np.random.Generator(np.random.PCG64(seed * 7919 + 1009 * s + 11))
        x = mu + 0.5 * sd * rng.standard_normal(A)
        for t in range(T):
            if t > 0:
                x = mu + rho * (x - mu) + walk * sd * rng.standard_normal(A)
            states[s, t] = _quantise(x).astype(np.float32)
        e = int(rng.integers(N))
        a = int(rng.integers(0, max(T // 2, 1)))
        b = min(T, a + max(T // 3, 1))
        omega[s, a:b, e] = elevate
        elevated[s] = e
        if latency_bounds:
            sla[s] = inst.sla[None, :]
    return Scenarios(states, sla, omega, elevated)


# ---------------------------------------------------------------------------
# Variant metadata of the full utility (Section II, Eq. 3)
# ---------------------------------------------------------------------------

MAX_VARIANTS = 4
Q_LLM = (1.000, 0.979)           # FP16, AWQ (relative perplexity)
Q_VIS = (0.73, 0.96, 1.00)       # YOLO11 n, s, m (mAP50-95, best = 1)
RELOAD_LLM, RELOAD_VIS = 30.0, 5.0


@dataclass
class Objective:
    variant: np.ndarray          # int32 [sum K]: variant of each option row
    n_variants: np.ndarray       # int32 [N]
    fmin: np.ndarray             # float32 [N][4]: per-variant throughput extremes
    fmax: np.ndarray             # float32 [N][4]
    quality: np.ndarray          # float32 [N][4]
    reload_cost: np.ndarray      # float32 [N]
    prev_variant: np.ndarray     # int32 [N]: variant deployed at the previous step (-1: none)
    tau: np.ndarray              # float32 [N]: floor on the normalised throughput
    alpha: float = 1.0 / 60.0
    beta: float = 5.0
    delta: float = 0.05


def make_objective(inst: Instance, seed: int = 0, tau_range=(0.2, 0.35), with_prev=True) -> Objective:
    """Draw the variant metadata for `inst`.  An option set is variants x
    runtime parameters (Section II), so option o of a model with K options
    and V variants belongs to variant (o V) // K.  LLMs have two variants,
    vision models three, with the quality values and reload costs the paper
    reports; the per-variant throughput extremes (profiling data in the paper)
    and the floors tau (a percentile of profiled performance in the paper)
    are drawn here around the surrogates' output scale."""
    rng = np.random.Generator(np.random.PCG64(seed * 7919 + 17))
    N = inst.n_models
    K = [int(k) for k in inst.n_options]
    variant = np.zeros(int(sum(K)), np.int32)
    nv = np.zeros(N, np.int32)
    fmin = np.zeros((N, MAX_VARIANTS), np.float32)
    fmax = np.ones((N, MAX_VARIANTS), np.float32)
    qual = np.zeros((N, MAX_VARIANTS), np.float32)
    cost = np.zeros(N, np.float32)
    prev = np.full(N, -1, np.int32)
    off = 0
    for i in range(N):
        llm = int(inst.model_type[i]) == 0
        q = Q_LLM if llm else Q_VIS
        V = min(len(q), K[i])
        nv[i] = V
        for o in range(K[i]):
            variant[off + o] = (o * V) // K[i]
        # extremes on the surrogate's output scale: sigmoid outputs lie in (0, 1)
        lo_r, hi_r = ((0.0, 0.2), (0.8, 1.0)) if inst.act == "sigmoid" else ((-2.0, -1.0), (1.0, 2.0))
        for v in range(V):
            qual[i, v] = q[len(q) - V + v]
            fmin[i, v] = _quantise(rng.uniform(*lo_r))
            fmax[i, v] = _quantise(rng.uniform(*hi_r))
        cost[i] = RELOAD_LLM if llm else RELOAD_VIS
        if with_prev:
            prev[i] = variant[off + int(rng.integers(0, K[i]))]
        off += K[i]
    tau = rng.uniform(tau_range[0], tau_range[1], N).astype(np.float32)
    return Objective(variant=variant, n_variants=nv, fmin=fmin, fmax=fmax, quality=qual, reload_cost=cost,
                     prev_variant=prev, tau=tau)


def linear_objective(inst: Instance) -> Objective:
    """Metadata under which the full utility equals sum_i omega_i thr_i and
    no floor binds: one variant, Q = 1, extremes (0, 1), no reload, no
    penalty."""
    N = inst.n_models
    fmax = np.ones((N, MAX_VARIANTS), np.float32)
    return Objective(variant=np.zeros(int(np.sum(inst.n_options)), np.int32), n_variants=np.ones(N, np.int32),
                     fmin=np.zeros((N, MAX_VARIANTS), np.float32), fmax=fmax,
                     quality=np.ones((N, MAX_VARIANTS), np.float32), reload_cost=np.zeros(N, np.float32),
                     prev_variant=np.full(N, -1, np.int32), tau=np.full(N, -np.inf, np.float32),
                     alpha=0.0, beta=0.0, delta=0.0)


@dataclass
class ProtocolDraws:
    """The random choices of the scheduling protocol (Section IV-C), drawn
    here so that every implementation of the protocol makes the same ones."""
    budget: np.ndarray           # uint64 [S][K_max]: uniform joint indices, StaticBudgetK's offline samples
    random: np.ndarray           # uint64 [S][T][R]: uniform joint indices, the Random scheduler's candidates
    ga_seed: np.ndarray          # uint64 [S][T]: the GA's generator key per decision


def protocol_draws(inst: Instance, n_scen: int, n_steps: int, seed: int = 0, k_max: int = 5000,
                   n_random: int = 64) -> ProtocolDraws:
    """Uniform joint indices for StaticBudgetK (the budgets use prefixes of
    one list) and candidates for the Random scheduler (it takes the first one
    that meets the VRAM cap), and one GA key per scenario and step."""
    rng = np.random.Generator(np.random.PCG64(seed * 104723 + 29))
    n = inst.space_size
    budget = rng.integers(0, n, (n_scen, k_max), dtype=np.uint64)
    rand = rng.integers(0, n, (n_scen, n_steps, n_random), dtype=np.uint64)
    ga_seed = rng.integers(0, 2 ** 62, (n_scen, n_steps), dtype=np.uint64)
    return ProtocolDraws(budget, rand, ga_seed)


@dataclass
class GAScenarios:
    sla: np.ndarray      # float32 [S][N]
    omega: np.ndarray    # float32 [S][N]


def ga_scenarios(n_models: int, n_scen: int = 64, seed: int = 0) -> GAScenarios:
    """Scenario s re-draws the per-model latency bounds U[0.5, 2.0] and the
    objective weights U[0.5, 1.5] from PCG64(seed*1000 + s)."""
    sla = np.zeros((n_scen, n_models), np.float32)
    om = np.zeros((n_scen, n_models), np.float32)
    for s in range(n_scen):
        r = np.random.Generator(np.random.PCG64(seed * 1000 + s))
        sla[s] = r.uniform(0.5, 2.0, n_models)
        om[s] = r.uniform(0.5, 1.5, n_models)
    return GAScenarios(sla=sla, omega=om)


@dataclass
class GAParams:
    n_scen: int = 64
    pop: int = 2048
    gens: int = 100          # offspring generations; (gens + 1) * pop evaluations per scenario
    tourn_k: int = 3
    p_cx: float = 0.7
    p_swap: float = 0.5
    p_mut: float = 0.05
    seed: int = 0


def cfg3(seed=0):
    """GA at N=5 on the N=5 instance: 64 scenarios, population 2048,
    100 generations, tournament 3, crossover 0.7 (uniform), mutation 0.05."""
    inst = cfg1(seed)
    inst.name = "ga_n5_s64_p2048_g100"
    return inst, ga_scenarios(inst.n_models, 64, seed), GAParams(seed=seed)


CONFIGS = {"cfg0": cfg0, "cfg1": cfg1, "cfg2": cfg2, "cfg4": cfg4}
