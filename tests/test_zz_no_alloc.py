"""mf_search_noalloc, the search entry point that allocates nothing (its
workspace is the library's fixed per-GPU scratch), against mf_search with a
caller workspace, both through the C ABI: two calls in a row on each
workload, the second on a smaller range, with identical results; requests
above the scratch size are refused before anything is enqueued."""
import ctypes as C

import numpy as np
import pytest

from paper_2609_02109_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2609_02109_amd import mf as m
    return m


def _args(mf, inst, lo, hi, k, state=None, worklist_cap=0):
    import torch
    d_sla = torch.as_tensor(inst.sla, device="cuda")
    d_om = torch.as_tensor(inst.omega, device="cuda")
    a = mf.SearchArgs(lo, hi, k, 0 if state is None else mf.MF_FIXED_STATE, d_sla.data_ptr(), d_om.data_ptr(),
                      None, None, mf.objective_args(None, inst.n_models))
    if state is not None:
        for t, v in enumerate(np.asarray(state, np.float32)):
            a.state[t] = float(v)
    a.worklist_cap = worklist_cap
    return a, (d_sla, d_om)


def _stream():
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _with_workspace(mf, p, a):
    import torch
    nb = C.c_size_t()
    assert mf.lib.mf_workspace_size(p.handle, C.byref(a), C.byref(nb)) == mf.MF_OK
    ws = torch.empty(max(nb.value, 256), dtype=torch.uint8, device="cuda")
    res = mf.Result()
    st = mf.lib.mf_search(p.handle, C.byref(a), C.c_void_p(ws.data_ptr()), ws.numel(), _stream(), C.byref(res))
    assert st == mf.MF_OK, mf.status_string(st)
    return res, nb.value


def _no_alloc(mf, p, a):
    res = mf.Result()
    st = mf.lib.mf_search_noalloc(p.handle, C.byref(a), _stream(), C.byref(res))
    assert st == mf.MF_OK, mf.status_string(st)
    return res


def _same(r, g):
    for f in ("n_eval", "n_vram", "n_feas", "n_flagged", "n_topk_collect", "n_top", "n_splits"):
        assert getattr(r, f) == getattr(g, f), f
    assert bytes(r.top_idx) == bytes(g.top_idx)
    assert bytes(r.top_J) == bytes(g.top_J)


CASES = [
    # (name, instance, k, state, (lo, hi) of the second, smaller call)
    ("n5", lambda: synth.cfg1(0), 16, False, (1_000, 61_000)),
    ("n6", lambda: synth.cfg2(0), 1, False, (5_000_000, 6_500_001)),
    ("n8_fixed_state", lambda: synth.cfg4(0), 64, True, (123_456_789, 1_123_456_789)),
]


@pytest.mark.parametrize("name,make,k,fixed,second", CASES, ids=[c[0] for c in CASES])
def test_no_alloc_search_matches_mf_search(mf, name, make, k, fixed, second):
    inst = make()
    print(f"no-alloc parity: {name}, |Lambda| = {inst.space_size}", flush=True)
    p = mf.Problem(inst)
    state = synth.make_state(inst, 0) if fixed else None
    for lo, hi in ((0, inst.space_size), second):
        a, keep = _args(mf, inst, lo, hi, k, state)
        g = _no_alloc(mf, p, a)
        r, nbytes = _with_workspace(mf, p, a)
        assert nbytes <= mf.NOALLOC_SCRATCH_BYTES
        _same(r, g)
        assert g.n_eval == hi - lo and g.n_top >= 1
        assert g.main_kernel_ms > 0.0


def test_no_alloc_refuses_requests_above_the_scratch(mf):
    # the N=8 bf16 search over 2^32 configurations with the default
    # certification list needs far more than the scratch; a bounded list fits
    inst = synth.cfg4(0)
    p = mf.Problem(inst)
    a, keep = _args(mf, inst, 0, inst.space_size, 64)
    nb = C.c_size_t()
    assert mf.lib.mf_workspace_size(p.handle, C.byref(a), C.byref(nb)) == mf.MF_OK
    assert nb.value > mf.NOALLOC_SCRATCH_BYTES
    res = mf.Result()
    assert mf.lib.mf_search_noalloc(p.handle, C.byref(a), _stream(), C.byref(res)) == mf.MF_ESCRATCH
    a.worklist_cap = 1 << 20
    assert mf.lib.mf_workspace_size(p.handle, C.byref(a), C.byref(nb)) == mf.MF_OK
    assert nb.value <= mf.NOALLOC_SCRATCH_BYTES
    assert mf.lib.mf_search_noalloc(p.handle, None, _stream(), C.byref(res)) == mf.MF_EINVAL
    assert mf.lib.mf_search_noalloc(p.handle, C.byref(a), _stream(), None) == mf.MF_EINVAL
    # after the refusals the scratch still serves a correct search
    small, keep2 = _args(mf, inst, 7, 300_007, 64)
    _same(_with_workspace(mf, p, small)[0], _no_alloc(mf, p, small))
