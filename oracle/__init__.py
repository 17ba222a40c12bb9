"""CPU oracle for the MeanField joint-configuration search (test infrastructure).

Only the tests, `__graft_entry__.smoke()` and the CPU-baseline leg of
`bench.py` may import this package.  It wraps `mf_oracle.c` (plain fp64
brute force; see that file's header for the definitions it follows) through
ctypes.  It imports nothing from the HIP library's package and shares no code
with it: instances arrive as duck-typed objects carrying numpy arrays.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mf_oracle.c")
GA_SRC = os.path.join(HERE, "mf_oracle_ga.c")
LIB = os.path.join(HERE, "libmf_oracle.so")
MAX_TOPK = 64


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (fp contraction off, explicit fma)."""
    srcs = [SRC] + ([GA_SRC] if os.path.exists(GA_SRC) else [])
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-march=x86-64-v3", "-std=c11",
           "-Wall", "-shared", "-fPIC", "-o", LIB + ".tmp", *srcs, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(LIB + ".tmp", LIB)
    return LIB


MAX_VARIANTS = 4


class _Obj(C.Structure):
    _fields_ = [("variant", C.c_void_p), ("fmin", C.c_void_p), ("fmax", C.c_void_p), ("quality", C.c_void_p),
                ("reload_cost", C.c_void_p), ("prev_variant", C.c_void_p), ("tau", C.c_void_p),
                ("alpha", C.c_float), ("beta", C.c_float), ("delta", C.c_float)]


class _Inst(C.Structure):
    _fields_ = [("n_models", C.c_int32), ("n_local", C.c_int32), ("n_agg", C.c_int32),
                ("hidden1", C.c_int32), ("hidden2", C.c_int32), ("bf16", C.c_int32),
                ("n_options", C.c_void_p), ("features", C.c_void_p), ("agg_cols", C.c_void_p),
                ("vram_slot", C.c_int32), ("vram_cap", C.c_float), ("weights", C.c_void_p),
                ("obj", C.c_void_p), ("fixed_state", C.c_void_p), ("raw_J", C.c_int32), ("sigmoid", C.c_int32)]


class _Result(C.Structure):
    _fields_ = [("n_eval", C.c_uint64), ("n_vram", C.c_uint64), ("n_feas", C.c_uint64),
                ("n_inexact_agg", C.c_uint64), ("n_near", C.c_uint64 * 4),
                ("n_top", C.c_int32), ("pad", C.c_int32),
                ("top_idx", C.c_uint64 * MAX_TOPK), ("top_J", C.c_double * MAX_TOPK)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        # MF_ORACLE_LIB names another build of the same sources (the
        # sanitizer test loads an ASan/UBSan build this way)
        path = os.environ.get("MF_ORACLE_LIB") or LIB
        if path == LIB and not os.path.exists(LIB):
            build()
        L = C.CDLL(path)
        P = C.c_void_p
        L.orc_space_size.restype = C.c_uint64
        L.orc_space_size.argtypes = [P]
        L.orc_decode.argtypes = [P, C.c_uint64, P]
        L.orc_encode.restype = C.c_uint64
        L.orc_encode.argtypes = [P, P]
        L.orc_aggregate.restype = C.c_int
        L.orc_aggregate.argtypes = [P, P, P]
        L.orc_eval.restype = C.c_int
        L.orc_eval.argtypes = [P, C.c_uint64, P, P, P, P, P, P]
        L.orc_search.restype = C.c_int
        L.orc_search.argtypes = [P, C.c_uint64, C.c_uint64, P, P, C.c_int, C.c_int, P, P, P, P]
        L.orc_eval_list.restype = C.c_int
        L.orc_eval_list.argtypes = [P, P, C.c_int64, P, P, C.c_int, P, P, P, P]
        L.orc_vram_feasible.restype = C.c_uint64
        L.orc_vram_feasible.argtypes = [P, P, C.c_uint64]
        L.orc_bf16_round.restype = C.c_double
        L.orc_bf16_round.argtypes = [C.c_double]
        for fn in ("orc_exp", "orc_sigmoid"):
            getattr(L, fn).restype = C.c_double
            getattr(L, fn).argtypes = [C.c_double]
        L.orc_philox4x64.argtypes = [P, P, P]
        L.orc_ga.restype = C.c_int
        L.orc_ga.argtypes = [P, P, P, P, P, P, P, C.c_int]
        L.orc_ga_next.restype = C.c_int
        L.orc_ga_next.argtypes = [P, P, C.c_int, C.c_int, P, P, P, C.c_uint64, P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


class Problem:
    """Holds contiguous copies of an instance's arrays and the C descriptor.
    `objective` (optional): an object with the arrays of the full utility of
    Eq. 3 (variant [sum K], fmin/fmax/quality [N][4], reload_cost [N],
    prev_variant [N], tau [N]) and alpha, beta, delta; None selects the
    linear objective.  `state` (optional): the observed aggregate state [A]
    fed to every surrogate, held fixed over the search (the paper's own
    semantics); None derives the aggregate from each candidate."""

    def __init__(self, inst, objective=None, state=None):
        self.n_options = np.ascontiguousarray(inst.n_options, dtype=np.int32)
        self.features = np.ascontiguousarray(inst.features, dtype=np.float32)
        self.agg_cols = np.ascontiguousarray(inst.agg_cols, dtype=np.int32)
        self.weights = np.ascontiguousarray(inst.weights, dtype=np.float32)
        self.N = int(self.n_options.shape[0])
        self.c = _Inst(self.N, int(inst.n_local), int(inst.n_agg), int(inst.hidden1),
                       int(inst.hidden2), 1 if inst.dtype == "bf16" else 0,
                       _ptr(self.n_options).value, _ptr(self.features).value,
                       _ptr(self.agg_cols).value, int(inst.vram_slot),
                       float(inst.vram_cap), _ptr(self.weights).value, None, None, 0,
                       1 if getattr(inst, "act", "identity") == "sigmoid" else 0)
        self.state = None
        if state is not None:
            self.state = np.ascontiguousarray(state, np.float32)
            self.c.fixed_state = _ptr(self.state).value
        self.obj = None
        if objective is not None:
            o = objective
            self._oa = [np.ascontiguousarray(o.variant, np.int32),
                        np.ascontiguousarray(o.fmin, np.float32).reshape(self.N, MAX_VARIANTS),
                        np.ascontiguousarray(o.fmax, np.float32).reshape(self.N, MAX_VARIANTS),
                        np.ascontiguousarray(o.quality, np.float32).reshape(self.N, MAX_VARIANTS),
                        np.ascontiguousarray(o.reload_cost, np.float32),
                        np.ascontiguousarray(o.prev_variant, np.int32),
                        np.ascontiguousarray(o.tau, np.float32)]
            self.obj = _Obj(*[_ptr(a).value for a in self._oa], float(o.alpha), float(o.beta), float(o.delta))
            self.c.obj = C.addressof(self.obj)
        self.ref = C.byref(self.c)

    @property
    def space_size(self) -> int:
        return int(lib().orc_space_size(self.ref))

    def decode(self, idx: int) -> np.ndarray:
        d = np.zeros(self.N, np.int32)
        lib().orc_decode(self.ref, C.c_uint64(idx), _ptr(d))
        return d

    def encode(self, digits) -> int:
        d = np.ascontiguousarray(digits, dtype=np.int32)
        return int(lib().orc_encode(self.ref, _ptr(d)))

    def aggregate(self, digits):
        d = np.ascontiguousarray(digits, dtype=np.int32)
        a = np.zeros(int(self.c.n_agg), np.float32)
        exact = lib().orc_aggregate(self.ref, _ptr(d), _ptr(a))
        return a, bool(exact)

    def eval(self, idx: int, sla, omega):
        sla = np.ascontiguousarray(sla, np.float32)
        om = np.ascontiguousarray(omega, np.float32)
        lat = np.zeros(self.N)
        thr = np.zeros(self.N)
        J = np.zeros(1)
        fl = np.zeros(1, np.uint32)
        lib().orc_eval(self.ref, C.c_uint64(idx), _ptr(sla), _ptr(om), _ptr(lat), _ptr(thr),
                       _ptr(J), _ptr(fl))
        return lat, thr, float(J[0]), int(fl[0])

    def search(self, sla, omega, k=1, lo=0, hi=None, threads=0, dump=False):
        """Brute force over [lo, hi).  Returns a dict with counts and top-k;
        with dump=True also per-config flags, J and (lat, thr) predictions."""
        if hi is None:
            hi = self.space_size
        sla = np.ascontiguousarray(sla, np.float32)
        om = np.ascontiguousarray(omega, np.float32)
        res = _Result()
        n = hi - lo
        fl = pr = jd = None
        if dump:
            fl = np.zeros(n, np.uint32)
            pr = np.zeros((n, self.N, 2), np.float64)
            jd = np.zeros(n, np.float64)
        rc = lib().orc_search(self.ref, C.c_uint64(lo), C.c_uint64(hi), _ptr(sla), _ptr(om),
                              int(k), int(threads), C.byref(res),
                              None if fl is None else _ptr(fl),
                              None if pr is None else _ptr(pr),
                              None if jd is None else _ptr(jd))
        if rc != 0:
            raise ValueError("orc_search rejected its arguments")
        nt = int(res.n_top)
        out = dict(n_eval=int(res.n_eval), n_vram=int(res.n_vram), n_feas=int(res.n_feas),
                   n_inexact_agg=int(res.n_inexact_agg), n_near=[int(x) for x in res.n_near],
                   top_idx=np.array(res.top_idx[:nt], np.uint64),
                   top_J=np.array(res.top_J[:nt], np.float64))
        if dump:
            out.update(flags=fl, pred=pr, J=jd)
        return out

    def eval_list(self, idx, sla, omega, threads=0, raw=False):
        """Evaluate an index list.  raw=True: J is the utility value also where
        a constraint fails (the flags say which)."""
        idx = np.ascontiguousarray(idx, np.uint64)
        n = int(idx.shape[0])
        sla = np.ascontiguousarray(sla, np.float32)
        om = np.ascontiguousarray(omega, np.float32)
        lat = np.zeros((n, self.N))
        thr = np.zeros((n, self.N))
        J = np.zeros(n)
        fl = np.zeros(n, np.uint32)
        self.c.raw_J = 1 if raw else 0
        try:
            lib().orc_eval_list(self.ref, _ptr(idx), n, _ptr(sla), _ptr(om), int(threads),
                                _ptr(lat), _ptr(thr), _ptr(J), _ptr(fl))
        finally:
            self.c.raw_J = 0
        return dict(lat=lat, thr=thr, J=J, flags=fl)

    def vram_feasible(self) -> np.ndarray:
        size = self.space_size
        buf = np.zeros(size, np.uint32)
        cnt = int(lib().orc_vram_feasible(self.ref, _ptr(buf), size))
        return buf[:cnt].copy()


class GAParams(C.Structure):
    _fields_ = [("n_scen", C.c_int32), ("pop", C.c_int32), ("gens", C.c_int32), ("tourn_k", C.c_int32),
                ("p_cx", C.c_float), ("p_swap", C.c_float), ("p_mut", C.c_float), ("pad", C.c_float),
                ("seed", C.c_uint64)]


def ga_params(n_scen, pop, gens, tourn_k=3, p_cx=0.7, p_swap=0.5, p_mut=0.05, seed=0):
    return GAParams(int(n_scen), int(pop), int(gens), int(tourn_k), float(p_cx), float(p_swap),
                    float(p_mut), 0.0, int(seed))


def _ga(self, sla, omega, pop=2048, gens=100, tourn_k=3, p_cx=0.7, p_swap=0.5, p_mut=0.05, seed=0,
        threads=0, final_pop=False):
    """GA replay (see mf_oracle_ga.c).  sla, omega: [S][N]."""
    sla = np.ascontiguousarray(sla, np.float32)
    om = np.ascontiguousarray(omega, np.float32)
    S = int(sla.shape[0])
    gp = ga_params(S, pop, gens, tourn_k, p_cx, p_swap, p_mut, seed)
    bi = np.zeros(S, np.uint64)
    bj = np.zeros(S, np.float64)
    fp = np.zeros((S, pop), np.uint64) if final_pop else None
    rc = lib().orc_ga(self.ref, C.byref(gp), _ptr(sla), _ptr(om), _ptr(bi), _ptr(bj),
                      None if fp is None else _ptr(fp), int(threads))
    if rc != 0:
        raise ValueError("orc_ga rejected its arguments")
    out = dict(best_idx=bi, best_J=bj)
    if final_pop:
        out["final_pop"] = fp
    return out


def _ga_next(self, s, g, pop_idx, fitness, feasible, pop, tourn_k=3, p_cx=0.7, p_swap=0.5, p_mut=0.05,
             seed=0):
    """One application of the GA operators (elitism, tournaments, crossover,
    mutation, repair) to a population with given fitness."""
    gp = ga_params(1, pop, 1, tourn_k, p_cx, p_swap, p_mut, seed)
    idx = np.ascontiguousarray(pop_idx, np.uint64)
    fit = np.ascontiguousarray(fitness, np.float64)
    fl = np.ascontiguousarray(feasible, np.uint32)
    out = np.zeros(pop, np.uint64)
    rc = lib().orc_ga_next(self.ref, C.byref(gp), int(s), int(g), _ptr(idx), _ptr(fit), _ptr(fl),
                           C.c_uint64(len(fl)), _ptr(out))
    if rc != 0:
        raise ValueError("orc_ga_next rejected its arguments")
    return out


Problem.ga = _ga
Problem.ga_next = _ga_next


def _step_objective(objective, t, n_models):
    # the deployment before step 0 is the objective's previous variants; a
    # static configuration is its own previous deployment afterwards (no
    # reload after step 0)
    if objective is None or t == 0:
        return objective
    from dataclasses import replace
    return replace(objective, prev_variant=np.full(n_models, -1, np.int32))


def static_eval(inst, objective, states, slas, omegas, idx, threads=0):
    """One configuration held over T steps (the static schedulers of Section
    IV-C, Table II).  Step t is the canonical evaluation with the step's
    observed state states[t] (Section III-B), bounds slas[t] and weights
    omegas[t].  Returns J [n][T] (the utility value, also where a constraint
    fails), flags [n][T] and S [n] = ((J_0 + J_1) + J_2) + ... in step order."""
    idx = np.ascontiguousarray(idx, np.uint64)
    T = len(states)
    N = int(inst.n_models)
    J = np.zeros((len(idx), T))
    F = np.zeros((len(idx), T), np.uint32)
    for t in range(T):
        r = Problem(inst, _step_objective(objective, t, N), state=states[t]).eval_list(
            idx, slas[t], omegas[t], threads=threads, raw=True)
        J[:, t] = r["J"]
        F[:, t] = r["flags"]
    S = J[:, 0].copy()
    for t in range(1, T):
        S = S + J[:, t]
    return J, F, S


def static_search(inst, objective, states, slas, omegas, k=1, lo=0, hi=None, threads=0):
    """argmax over [lo, hi) of S(lambda) = sum_t J_t(lambda) among the
    configurations feasible at every step (VRAM cap once; every step's
    latency bounds and floors); top-k by (S desc, index asc)."""
    if hi is None:
        hi = int(np.prod([int(x) for x in inst.n_options], dtype=object))
    idx = np.arange(lo, hi, dtype=np.uint64)
    J, F, S = static_eval(inst, objective, states, slas, omegas, idx, threads)
    vram = (F[:, 0] & FLAG_VRAM) != 0
    svc = np.all((F & FLAG_SLA) != 0, axis=1)
    feas = vram & svc
    sel = np.flatnonzero(feas)
    order = np.lexsort((idx[sel], -S[sel]))[:k]
    flags = vram.astype(np.uint32) | (svc.astype(np.uint32) << 1) | (feas.astype(np.uint32) << 2)
    return dict(n_vram=int(vram.sum()), n_feas=int(feas.sum()), top_idx=idx[sel][order],
                top_J=S[sel][order], flags=flags, S=S, J=J, step_flags=F)


def philox4x64(ctr, key):
    c = np.ascontiguousarray(ctr, np.uint64)
    k = np.ascontiguousarray(key, np.uint64)
    o = np.zeros(4, np.uint64)
    lib().orc_philox4x64(_ptr(c), _ptr(k), _ptr(o))
    return [int(x) for x in o]


def bf16_round(x: float) -> float:
    return float(lib().orc_bf16_round(float(x)))


def exp(x: float) -> float:
    """The oracle's e^x (|x| <= 700; the algorithm of mf_oracle.c)."""
    return float(lib().orc_exp(float(x)))


def sigmoid(y: float) -> float:
    return float(lib().orc_sigmoid(float(y)))


FLAG_VRAM, FLAG_SLA, FLAG_FEAS, FLAG_EXACT = 1, 2, 4, 8
