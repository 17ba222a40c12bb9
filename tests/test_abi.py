"""C ABI: the library loads and exports every function include/mf.h declares,
and argument validation needs no GPU.  No compute calls (CPU-only test)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "mf.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mf_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ["mf_problem_create", "mf_problem_destroy", "mf_search", "mf_workspace_size",
              "mf_eval_fast", "mf_eval_canonical", "mf_ga_run", "mf_ga_workspace_size",
              "mf_decode", "mf_space_size", "mf_status_string"]:
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2609_02109_amd import mf
    for n in declared_functions():
        assert hasattr(mf.lib, n), f"{n} declared in mf.h but not exported by libmf.so"
    assert sorted(mf.EXPORTS) == declared_functions()


def test_status_strings():
    from paper_2609_02109_amd import mf
    for s in range(7):
        assert mf.status_string(s).startswith("MF_")
    assert "unknown" in mf.status_string(99)


def test_create_rejects_bad_descriptors_before_any_device_call():
    from paper_2609_02109_amd import mf
    import numpy as np
    K = np.array([3, 4], np.int32)
    cols = np.array([3, 4, 5, 0], np.int32)
    dummy = np.zeros(16, np.float32)

    def create(**over):
        d = dict(n_models=2, n_local=8, n_agg=4, hidden1=32, hidden2=32, h_n_options=K.ctypes.data,
                 h_agg_cols=cols.ctypes.data, vram_slot=1, vram_cap=80.0, dtype=mf.MF_F32)
        d.update(over)
        desc = mf.Desc(**d)
        h = C.c_void_p()
        return mf.lib.mf_problem_create(C.byref(desc), dummy.ctypes.data_as(C.c_void_p),
                                        dummy.ctypes.data_as(C.c_void_p), None, C.byref(h))
    bad_k = np.array([3, 0], np.int32)
    bad_cols = np.array([3, 4, 5, 9], np.int32)
    assert create(n_models=0) == mf.MF_EINVAL
    assert create(n_models=17) == mf.MF_EINVAL
    assert create(h_n_options=None) == mf.MF_EINVAL
    assert create(h_n_options=bad_k.ctypes.data) == mf.MF_EINVAL
    assert create(h_agg_cols=bad_cols.ctypes.data) == mf.MF_EINVAL
    assert create(vram_slot=4) == mf.MF_EINVAL
    assert create(vram_cap=float("nan")) == mf.MF_EINVAL
    assert create(dtype=7) == mf.MF_EINVAL
    assert create(hidden1=0) == mf.MF_EINVAL
    big = np.full(9, 255, np.int32)
    assert create(n_models=9, h_n_options=big.ctypes.data) == mf.MF_EOVERFLOW
    assert mf.lib.mf_problem_create(None, None, None, None, None) == mf.MF_EINVAL


def test_null_handles_rejected():
    from paper_2609_02109_amd import mf
    out = C.c_uint64()
    assert mf.lib.mf_space_size(None, C.byref(out)) == mf.MF_EINVAL
    assert mf.lib.mf_search(None, None, None, 0, None, None) == mf.MF_EINVAL
    assert mf.lib.mf_eval_fast(None, None, 0, None, None) == mf.MF_EINVAL
    assert mf.lib.mf_ga_run(None, None, None, 0, None, None, None, None) == mf.MF_EINVAL
    mf.lib.mf_problem_destroy(None)
