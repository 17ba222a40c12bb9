"""ctypes binding of libmf.so (include/mf.h).

Marshalling only: torch tensors supply device memory and the HIP stream;
every step of the search runs in the library's kernels.  Importing this module
fails loudly when the HIP library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
import threading

import numpy as np
# torch first: it brings the HIP runtime it was built against, and the
# library then binds to that same runtime (one runtime per process; loading
# the library first would pull in another copy that torch then reuses)
import torch  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmf.so")

MF_OK, MF_EINVAL, MF_ENOMEM, MF_EDEVICE, MF_EUNSUPPORTED, MF_EOVERFLOW, MF_EINTERNAL, MF_ESCRATCH = range(8)
NOALLOC_SCRATCH_BYTES = 128 << 20
MF_F32, MF_BF16 = 0, 1
MF_ACT_IDENTITY, MF_ACT_SIGMOID = 0, 1
MF_DUMP = 1
MF_FIXED_STATE = 2
MAX_AGG = 16
MAX_TOPK = 64
MAX_MODELS = 16

EXPORTS = ["mf_problem_bytes", "mf_problem_create", "mf_problem_destroy", "mf_space_size", "mf_decode",
           "mf_workspace_size", "mf_search", "mf_search_noalloc", "mf_eval_fast", "mf_eval_canonical",
           "mf_static_workspace_size", "mf_search_static", "mf_eval_static",
           "mf_ga_workspace_size", "mf_ga_run", "mf_status_string"]


class MfError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)}")
        self.status = status


MAX_VARIANTS = 4
MF_OBJ_LINEAR, MF_OBJ_EQ3 = 0, 1


class Variants(C.Structure):
    _fields_ = [("h_variant", C.c_void_p), ("h_n_variants", C.c_void_p), ("h_fmin", C.c_void_p),
                ("h_fmax", C.c_void_p), ("h_quality", C.c_void_p), ("h_reload_cost", C.c_void_p)]


class Desc(C.Structure):
    _fields_ = [("n_models", C.c_int32), ("n_local", C.c_int32), ("n_agg", C.c_int32),
                ("hidden1", C.c_int32), ("hidden2", C.c_int32),
                ("h_n_options", C.c_void_p), ("h_agg_cols", C.c_void_p),
                ("vram_slot", C.c_int32), ("vram_cap", C.c_float), ("dtype", C.c_int32),
                ("variants", C.c_void_p), ("output_act", C.c_int32)]


class Objective(C.Structure):
    _fields_ = [("kind", C.c_int32), ("alpha", C.c_float), ("beta", C.c_float), ("delta", C.c_float),
                ("tau", C.c_float * MAX_MODELS), ("prev_variant", C.c_int32 * MAX_MODELS)]


class SearchArgs(C.Structure):
    _fields_ = [("lo", C.c_uint64), ("hi", C.c_uint64), ("top_k", C.c_int32), ("flags", C.c_uint32),
                ("d_sla", C.c_void_p), ("d_omega", C.c_void_p), ("d_mask", C.c_void_p),
                ("d_pred", C.c_void_p), ("objective", Objective), ("state", C.c_float * MAX_AGG),
                ("worklist_cap", C.c_uint32)]


def objective_args(obj, n_models: int) -> Objective:
    """mf_objective for a search: None -> the linear objective; otherwise an
    object with alpha, beta, delta, tau [N] and prev_variant [N] (Eq. 3)."""
    o = Objective()
    if obj is None:
        return o
    o.kind = MF_OBJ_EQ3
    o.alpha, o.beta, o.delta = float(obj.alpha), float(obj.beta), float(obj.delta)
    for i in range(n_models):
        o.tau[i] = float(obj.tau[i])
        o.prev_variant[i] = int(obj.prev_variant[i])
    return o


class Result(C.Structure):
    _fields_ = [("n_eval", C.c_uint64), ("n_vram", C.c_uint64), ("n_feas", C.c_uint64),
                ("n_flagged", C.c_uint64), ("n_topk_collect", C.c_uint64),
                ("n_top", C.c_int32), ("n_splits", C.c_int32),
                ("top_idx", C.c_uint64 * MAX_TOPK), ("top_J", C.c_double * MAX_TOPK),
                ("main_kernel_ms", C.c_float), ("pad", C.c_float)]


MAX_STEPS = 32


class StaticArgs(C.Structure):
    _fields_ = [("lo", C.c_uint64), ("hi", C.c_uint64), ("top_k", C.c_int32), ("n_steps", C.c_int32),
                ("d_sla", C.c_void_p), ("d_omega", C.c_void_p), ("h_state", C.c_void_p),
                ("objective", Objective), ("d_mask", C.c_void_p)]


class GAArgs(C.Structure):
    _fields_ = [("n_scen", C.c_int32), ("pop", C.c_int32), ("gens", C.c_int32), ("tourn_k", C.c_int32),
                ("p_cx", C.c_float), ("p_swap", C.c_float), ("p_mut", C.c_float), ("pad", C.c_float),
                ("seed", C.c_uint64), ("d_sla", C.c_void_p), ("d_omega", C.c_void_p),
                ("flags", C.c_uint32), ("state", C.c_float * MAX_AGG), ("objective", Objective),
                ("h_forwards", C.c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2609_02109_amd.build` (or __graft_entry__.build())")
    L = C.CDLL(LIB_PATH)
    P = C.c_void_p
    S = C.c_int
    sig = {
        "mf_problem_bytes": (S, [P, P]),
        "mf_problem_create": (S, [P, P, P, P, C.c_size_t, P, P]),
        "mf_problem_destroy": (None, [P]),
        "mf_space_size": (S, [P, P]),
        "mf_decode": (S, [P, C.c_uint64, P]),
        "mf_workspace_size": (S, [P, P, P]),
        "mf_search": (S, [P, P, P, C.c_size_t, P, P]),
        "mf_search_noalloc": (S, [P, P, P, P]),
        "mf_eval_fast": (S, [P, P, C.c_int64, P, P]),
        "mf_eval_canonical": (S, [P, P, C.c_int64, P, P, P, P, P, P]),
        "mf_static_workspace_size": (S, [P, P, P]),
        "mf_search_static": (S, [P, P, P, C.c_size_t, P, P]),
        "mf_eval_static": (S, [P, P, P, C.c_int64, P, P, P, P, C.c_size_t, P]),
        "mf_ga_workspace_size": (S, [P, P, P]),
        "mf_ga_run": (S, [P, P, P, C.c_size_t, P, P, P, P]),
        "mf_status_string": (C.c_char_p, [S]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


lib = _load()


def status_string(s: int) -> str:
    return lib.mf_status_string(int(s)).decode()


def _check(s: int, where: str):
    if s != MF_OK:
        raise MfError(s, where)


def _ptr(t):
    """Device (or host) address of a torch tensor or numpy array; None -> NULL."""
    if t is None:
        return None
    if hasattr(t, "data_ptr"):
        return C.c_void_p(t.data_ptr())
    return t.ctypes.data_as(C.c_void_p)


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _keep_for(stream, *tensors):
    """Tensors read or written by work enqueued on `stream`: when that is not
    torch's current stream, tell the caching allocator, so that their memory
    is not handed out again before that work has run."""
    if stream is None or stream == torch.cuda.current_stream():
        return
    for t in tensors:
        if isinstance(t, torch.Tensor) and t.is_cuda:
            t.record_stream(stream)


class Problem:
    """A created problem (mf_problem).  `inst` carries the instance arrays
    (n_options, features, agg_cols, weights, ...), e.g. a synth.Instance."""

    def __init__(self, inst, device="cuda", stream=None, variants=None):
        self.inst = inst
        self.N = int(inst.n_models)
        self.A = int(inst.n_agg)
        self.device = torch.device(device)
        self._n_options = np.ascontiguousarray(inst.n_options, np.int32)
        self._agg_cols = np.ascontiguousarray(inst.agg_cols, np.int32)
        feats = torch.from_numpy(np.ascontiguousarray(inst.features, np.float32)).to(self.device)
        w = torch.from_numpy(np.ascontiguousarray(inst.weights, np.float32)).to(self.device)
        self._var = None
        if variants is not None:
            # static variant metadata of Eq. 3 (variant per option row,
            # per-variant extremes and quality, reload cost per model)
            v = variants
            self._var_arrays = [np.ascontiguousarray(v.variant, np.int32),
                                np.ascontiguousarray(v.n_variants, np.int32),
                                np.ascontiguousarray(v.fmin, np.float32).reshape(self.N, MAX_VARIANTS),
                                np.ascontiguousarray(v.fmax, np.float32).reshape(self.N, MAX_VARIANTS),
                                np.ascontiguousarray(v.quality, np.float32).reshape(self.N, MAX_VARIANTS),
                                np.ascontiguousarray(v.reload_cost, np.float32)]
            self._var = Variants(*[_ptr(a).value for a in self._var_arrays])
        self.desc = Desc(self.N, int(inst.n_local), int(inst.n_agg), int(inst.hidden1),
                         int(inst.hidden2), _ptr(self._n_options), _ptr(self._agg_cols),
                         int(inst.vram_slot), float(inst.vram_cap),
                         MF_BF16 if inst.dtype == "bf16" else MF_F32,
                         C.addressof(self._var) if self._var is not None else None,
                         MF_ACT_SIGMOID if getattr(inst, "act", "identity") == "sigmoid" else MF_ACT_IDENTITY)
        # the problem's tables live in a caller-owned device buffer, kept
        # alive as long as the problem
        nb = C.c_size_t()
        _check(lib.mf_problem_bytes(C.byref(self.desc), C.byref(nb)), "mf_problem_bytes")
        self._tables = torch.empty(max(int(nb.value), 256), dtype=torch.uint8, device=self.device)
        _keep_for(stream, feats, w, self._tables)
        h = C.c_void_p()
        _check(lib.mf_problem_create(C.byref(self.desc), _ptr(feats), _ptr(w), _ptr(self._tables),
                                     C.c_size_t(self._tables.numel()), _stream(stream), C.byref(h)),
               "mf_problem_create")
        self.handle = h
        # one workspace per (thread, stream): calls that overlap must not share one
        self._ws = {}
        self._ws_lock = threading.Lock()

    def close(self):
        if getattr(self, "handle", None):
            lib.mf_problem_destroy(self.handle)
            self.handle = None
            self._tables = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def space_size(self) -> int:
        out = C.c_uint64()
        _check(lib.mf_space_size(self.handle, C.byref(out)), "mf_space_size")
        return int(out.value)

    def decode(self, idx: int) -> np.ndarray:
        d = np.zeros(self.N, np.int32)
        _check(lib.mf_decode(self.handle, C.c_uint64(idx), _ptr(d)), "mf_decode")
        return d

    def _dev(self, a, dtype):
        if a is None:
            return None
        if isinstance(a, torch.Tensor):
            return a.to(self.device, dtype).contiguous()
        return torch.as_tensor(np.asarray(a), dtype=dtype, device=self.device).contiguous()

    def workspace(self, nbytes: int, stream=None):
        """A device workspace of at least nbytes for calls from this thread on
        `stream` (None: torch's current stream)."""
        s = stream if stream is not None else torch.cuda.current_stream()
        key = (threading.get_ident(), s.cuda_stream)
        with self._ws_lock:
            ws = self._ws.get(key)
            if ws is None or ws.numel() < nbytes:
                ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
                _keep_for(stream, ws)
                self._ws[key] = ws
        return ws

    def search(self, sla, omega, k=1, lo=0, hi=None, dump=False, stream=None, objective=None, state=None,
               worklist_cap=0):
        """Exhaustive search over [lo, hi).  Returns a dict of counts and the
        exact top-k; with dump=True also the per-index mask and fast-path
        predictions (device tensors).  objective: None (linear) or an object
        with alpha, beta, delta, tau, prev_variant (Eq. 3; the problem must
        have been created with variants).  state: None (each candidate's own
        aggregate feeds the surrogates) or the observed aggregate [A] held
        fixed for the whole search (Section III-B).  worklist_cap: bound on
        the certification list (0: the library's default)."""
        if hi is None:
            hi = self.space_size
        d_sla = self._dev(sla, torch.float32)
        d_om = self._dev(omega, torch.float32)
        mask = pred = None
        if dump:
            mask = torch.zeros(max(hi - lo, 1), dtype=torch.uint8, device=self.device)
            pred = torch.zeros((max(hi - lo, 1), self.N, 2), dtype=torch.float32, device=self.device)
        flags = (MF_DUMP if dump else 0) | (MF_FIXED_STATE if state is not None else 0)
        args = SearchArgs(lo, hi, int(k), flags, _ptr(d_sla), _ptr(d_om),
                          _ptr(mask), _ptr(pred), objective_args(objective, self.N))
        args.worklist_cap = int(worklist_cap)
        if state is not None:
            st = np.asarray(state, np.float32).reshape(-1)
            if st.size != self.A:
                raise ValueError(f"state has {st.size} values, the problem {self.A} aggregate slots")
            for t in range(st.size):
                args.state[t] = float(st[t])
        nbytes = C.c_size_t()
        _check(lib.mf_workspace_size(self.handle, C.byref(args), C.byref(nbytes)), "mf_workspace_size")
        ws = self.workspace(nbytes.value, stream)
        _keep_for(stream, d_sla, d_om, mask, pred)
        res = Result()
        _check(lib.mf_search(self.handle, C.byref(args), _ptr(ws), C.c_size_t(ws.numel()),
                             _stream(stream), C.byref(res)), "mf_search")
        nt = int(res.n_top)
        out = dict(n_eval=int(res.n_eval), n_vram=int(res.n_vram), n_feas=int(res.n_feas),
                   n_flagged=int(res.n_flagged), n_topk_collect=int(res.n_topk_collect),
                   n_splits=int(res.n_splits), main_kernel_ms=float(res.main_kernel_ms),
                   top_idx=np.array(res.top_idx[:nt], np.uint64),
                   top_J=np.array(res.top_J[:nt], np.float64))
        if dump:
            out.update(mask=mask[:hi - lo], pred=pred[:hi - lo])
        return out

    def _static_args(self, states, slas, omegas, objective, k=1, lo=0, hi=None, mask=None, stream=None):
        st = np.ascontiguousarray(states, np.float32).reshape(-1, self.A)
        T = int(st.shape[0])
        d_sla = self._dev(np.asarray(slas, np.float32).reshape(T, self.N), torch.float32)
        d_om = self._dev(np.asarray(omegas, np.float32).reshape(T, self.N), torch.float32)
        args = StaticArgs(int(lo), int(self.space_size if hi is None else hi), int(k), T, _ptr(d_sla), _ptr(d_om),
                          _ptr(st), objective_args(objective, self.N), _ptr(mask))
        nbytes = C.c_size_t()
        _check(lib.mf_static_workspace_size(self.handle, C.byref(args), C.byref(nbytes)), "mf_static_workspace_size")
        return args, self.workspace(nbytes.value, stream), (st, d_sla, d_om)

    def search_static(self, states, slas, omegas, k=1, lo=0, hi=None, objective=None, dump=False, stream=None):
        """One configuration held over T steps (states [T][A], slas and omegas
        [T][N]): the exact top-k of S = sum_t J_t among the configurations
        feasible at every step; with dump=True also the per-index mask."""
        if hi is None:
            hi = self.space_size
        mask = torch.zeros(max(hi - lo, 1), dtype=torch.uint8, device=self.device) if dump else None
        args, ws, keep = self._static_args(states, slas, omegas, objective, k, lo, hi, mask, stream)
        _keep_for(stream, mask, *keep[1:])
        res = Result()
        _check(lib.mf_search_static(self.handle, C.byref(args), _ptr(ws), C.c_size_t(ws.numel()), _stream(stream),
                                    C.byref(res)), "mf_search_static")
        nt = int(res.n_top)
        out = dict(n_eval=int(res.n_eval), n_vram=int(res.n_vram), n_feas=int(res.n_feas),
                   main_kernel_ms=float(res.main_kernel_ms), top_idx=np.array(res.top_idx[:nt], np.uint64),
                   top_J=np.array(res.top_J[:nt], np.float64))
        if dump:
            out["mask"] = mask[:hi - lo]
        return out

    def eval_static(self, idx, states, slas, omegas, objective=None, stream=None):
        """Per-step utilities of an index list held over T steps: J [n][T],
        S [n] (step-order sum), flags [n][T] (bit0 VRAM, bit1 the step's
        service constraints)."""
        d_idx = self._dev(np.asarray(idx, np.uint64).astype(np.int64), torch.int64)
        n = int(d_idx.numel())
        args, ws, keep = self._static_args(states, slas, omegas, objective, stream=stream)
        T = int(args.n_steps)
        J = torch.zeros((max(n, 1), T), dtype=torch.float64, device=self.device)
        S = torch.zeros(max(n, 1), dtype=torch.float64, device=self.device)
        F = torch.zeros((max(n, 1), T), dtype=torch.int32, device=self.device)
        _keep_for(stream, d_idx, J, S, F, *keep[1:])
        _check(lib.mf_eval_static(self.handle, C.byref(args), _ptr(d_idx), n, _ptr(J), _ptr(S), _ptr(F), _ptr(ws),
                                  C.c_size_t(ws.numel()), _stream(stream)), "mf_eval_static")
        return dict(J=J[:n].cpu().numpy(), S=S[:n].cpu().numpy(), flags=F[:n].cpu().numpy().astype(np.uint32))

    def search_raw(self, args: SearchArgs, ws, stream=None) -> Result:
        """Direct call for timing loops: caller-built SearchArgs and workspace."""
        res = Result()
        _check(lib.mf_search(self.handle, C.byref(args), _ptr(ws), C.c_size_t(ws.numel()),
                             _stream(stream), C.byref(res)), "mf_search")
        return res

    def eval_fast(self, idx, stream=None):
        d_idx = self._dev(idx, torch.int64)
        n = int(d_idx.numel())
        pred = torch.zeros((max(n, 1), self.N, 2), dtype=torch.float32, device=self.device)
        _keep_for(stream, d_idx, pred)
        _check(lib.mf_eval_fast(self.handle, _ptr(d_idx), n, _ptr(pred), _stream(stream)),
               "mf_eval_fast")
        return pred[:n]

    def eval_canonical(self, idx, sla, omega, stream=None):
        d_idx = self._dev(idx, torch.int64)
        n = int(d_idx.numel())
        pred = torch.zeros((max(n, 1), self.N, 2), dtype=torch.float64, device=self.device)
        J = torch.zeros(max(n, 1), dtype=torch.float64, device=self.device)
        fl = torch.zeros(max(n, 1), dtype=torch.int32, device=self.device)
        d_sla = self._dev(sla, torch.float32)
        d_om = self._dev(omega, torch.float32)
        _keep_for(stream, d_idx, d_sla, d_om, pred, J, fl)
        _check(lib.mf_eval_canonical(self.handle, _ptr(d_idx), n, _ptr(d_sla), _ptr(d_om), _ptr(pred),
                                     _ptr(J), _ptr(fl), _stream(stream)), "mf_eval_canonical")
        return dict(pred=pred[:n], J=J[:n], flags=fl[:n])

    def ga(self, sla, omega, pop=2048, gens=100, tourn_k=3, p_cx=0.7, p_swap=0.5, p_mut=0.05,
           seed=0, final_pop=False, stream=None, objective=None, state=None):
        """GA scheduler over S scenarios (rows of sla / omega); objective and
        state as in search()."""
        d_sla = self._dev(sla, torch.float32)
        d_om = self._dev(omega, torch.float32)
        S = int(d_sla.shape[0])
        args = GAArgs(S, int(pop), int(gens), int(tourn_k), float(p_cx), float(p_swap), float(p_mut),
                      0.0, int(seed), _ptr(d_sla), _ptr(d_om))
        args.objective = objective_args(objective, self.N)
        if state is not None:
            st = np.asarray(state, np.float32).reshape(-1)
            if st.size != self.A:
                raise ValueError(f"state has {st.size} values, the problem {self.A} aggregate slots")
            args.flags = MF_FIXED_STATE
            for t in range(st.size):
                args.state[t] = float(st[t])
        nbytes = C.c_size_t()
        _check(lib.mf_ga_workspace_size(self.handle, C.byref(args), C.byref(nbytes)),
               "mf_ga_workspace_size")
        ws = self.workspace(nbytes.value, stream)
        best_idx = np.zeros(S, np.uint64)
        best_J = np.zeros(S, np.float64)
        forwards = np.zeros(1, np.uint64)
        args.h_forwards = _ptr(forwards)
        fp = torch.zeros((S, pop), dtype=torch.int64, device=self.device) if final_pop else None
        _keep_for(stream, d_sla, d_om, fp)
        _check(lib.mf_ga_run(self.handle, C.byref(args), _ptr(ws), C.c_size_t(ws.numel()),
                             _stream(stream), _ptr(best_idx), _ptr(best_J), _ptr(fp)), "mf_ga_run")
        out = dict(best_idx=best_idx, best_J=best_J, forwards=int(forwards[0]))
        if final_pop:
            out["final_pop"] = fp
        return out
