"""GPU parity of the exhaustive search against the CPU oracle (through the C ABI).

Bars (tiers):
  1. digits, aggregate, VRAM mask, n_vram: bit-exact.
  2. fast-path fp32 predictions: |gpu - oracle| <= 1e-5 * max(|oracle|, rms)
     where rms is the root mean square of that output over the checked set
     (a relative bar that does not blow up at outputs crossing zero).
  3. latency masks, feasible mask, n_feas, top-k indices and canonical J:
     bit-exact (the GPU re-evaluates undecidable cases with the same fp64
     chain the oracle uses).
"""
import json
import math
import os

import numpy as np
import pytest

from paper_2609_02109_amd import synth

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TOL_F32 = 1e-5


@pytest.fixture(scope="module")
def mf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_02109_amd import mf as mfmod
    return mfmod


def check_predictions(pred_gpu, pred_ref, tol=TOL_F32):
    g = np.asarray(pred_gpu, np.float64)
    r = np.asarray(pred_ref, np.float64)
    for o in range(2):
        rms = math.sqrt(float(np.mean(r[..., o] ** 2)))
        err = np.abs(g[..., o] - r[..., o])
        lim = tol * np.maximum(np.abs(r[..., o]), rms)
        bad = err > lim
        assert not bad.any(), f"output {o}: {int(bad.sum())} predictions off, worst {float(err.max()):.3e}"


def run_range_parity(mf, orc, inst, lo, hi, k, tol=TOL_F32):
    print(f"[parity] {inst.name} seed={inst.seed} range=[{lo},{hi}) k={k}", flush=True)
    p = mf.Problem(inst)
    g = p.search(inst.sla, inst.omega, k=k, lo=lo, hi=hi, dump=True)
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=k, lo=lo, hi=hi, dump=True)
    assert g["n_eval"] == hi - lo
    assert g["n_vram"] == r["n_vram"]
    assert g["n_feas"] == r["n_feas"]
    gm = g["mask"].cpu().numpy().astype(np.uint32)
    rf = r["flags"]
    np.testing.assert_array_equal(gm & 1, rf & 1)             # VRAM mask
    np.testing.assert_array_equal((gm >> 1) & 1, (rf >> 1) & 1)  # every latency bound
    np.testing.assert_array_equal((gm >> 2) & 1, (rf >> 2) & 1)  # feasible
    np.testing.assert_array_equal(g["top_idx"], r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()
    check_predictions(g["pred"].cpu().numpy(), r["pred"], tol=tol)
    p.close()
    return g, r


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_cfg0_full(mf, orc, seed):
    inst = synth.cfg0(seed)
    run_range_parity(mf, orc, inst, 0, inst.space_size, 1)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_cfg1_full(mf, orc, seed):
    inst = synth.cfg1(seed)
    g, _ = run_range_parity(mf, orc, inst, 0, inst.space_size, 16)
    gold = json.load(open(os.path.join(GOLDEN, f"cfg1_s{seed}.json")))
    assert gold["n_feas"] == g["n_feas"] and gold["top_idx"] == [int(x) for x in g["top_idx"]]


@pytest.mark.parametrize("k", [16, 64])
def test_cfg1_small_range_finish(mf, orc, k):
    # the N=5 space takes the small-range path: each fast workgroup keeps its
    # k best canonical keys and one workgroup finishes; 206 workgroups x 16
    # keys are staged in LDS by the finish kernel, 206 x 64 exceed its LDS
    # limit and are read from global memory
    inst = synth.cfg1(1)
    print(f"[small-range] cfg1 seed=1 k={k}", flush=True)
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=k)
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=k)
    assert g["n_vram"] == r["n_vram"] and g["n_feas"] == r["n_feas"]
    np.testing.assert_array_equal(g["top_idx"], r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_tight_latency_bounds(mf, orc):
    # bounds drawn near the latency distribution: every model's bound binds
    # for a large share of configurations, so many decisions go to the
    # canonical re-evaluation
    inst = synth.make_instance([12, 12, 9, 9, 9], seed=5, vram_quantile=0.75,
                               sla_range=(-0.15, 0.15), top_k=16)
    g, r = run_range_parity(mf, orc, inst, 0, inst.space_size, 16)
    assert g["n_flagged"] > 0
    assert 0 < r["n_feas"] < r["n_vram"]


def test_cfg2_ragged_ranges(mf, orc):
    inst = synth.cfg2(0)
    run_range_parity(mf, orc, inst, 0, 1 << 18, 1)
    run_range_parity(mf, orc, inst, 123_457, 123_457 + 300_001, 4)
    n = inst.space_size
    run_range_parity(mf, orc, inst, n - 70_001, n, 8)   # ragged tail of the space


def test_cfg2_full_against_golden(mf):
    path = os.path.join(GOLDEN, "cfg2_s0.json")
    if not os.path.exists(path):
        pytest.skip("golden cfg2_s0.json not generated")
    gold = json.load(open(path))
    inst = synth.cfg2(0)
    print(f"[parity] cfg2 full space {inst.space_size}", flush=True)
    p = mf.Problem(inst)
    g = p.search(inst.sla, inst.omega, k=16)
    assert g["n_vram"] == gold["n_vram"]
    assert g["n_feas"] == gold["n_feas"]
    assert [int(x) for x in g["top_idx"]] == gold["top_idx"]
    assert [float(x).hex() for x in g["top_J"]] == gold["top_J"]


@pytest.mark.parametrize("shape", [
    dict(n_options=[5], n_local=8, n_agg=4, hidden=32),               # N = 1
    dict(n_options=[1, 7, 1, 3], n_local=8, n_agg=2, hidden=32),       # options count 1
    dict(n_options=[3, 4, 5], n_local=12, n_agg=8, hidden=64),
    dict(n_options=[2] * 16, n_local=8, n_agg=6, hidden=32),           # N = 16
    dict(n_options=[255, 3], n_local=8, n_agg=4, hidden=64),           # widest option set
])
def test_shapes(mf, orc, shape):
    inst = synth.make_instance(shape["n_options"], shape["n_local"], shape["n_agg"], shape["hidden"],
                               shape["hidden"], seed=3, vram_quantile=0.6, sla_range=(-0.2, 0.8))
    run_range_parity(mf, orc, inst, 0, inst.space_size, 5)


def test_degenerate_cases(mf, orc):
    inst = synth.cfg1(0)
    p = mf.Problem(inst)
    # empty range
    g = p.search(inst.sla, inst.omega, k=3, lo=100, hi=100)
    assert g["n_eval"] == 0 and g["n_feas"] == 0 and len(g["top_idx"]) == 0
    # single configuration
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=3, lo=777, hi=778)
    g = p.search(inst.sla, inst.omega, k=3, lo=777, hi=778)
    assert g["n_feas"] == r["n_feas"] and list(g["top_idx"]) == list(r["top_idx"])
    # nothing feasible: cap below every VRAM sum
    inst2 = synth.cfg1(0)
    inst2.vram_cap = 1.0
    p2 = mf.Problem(inst2)
    g = p2.search(inst2.sla, inst2.omega, k=16)
    assert g["n_vram"] == 0 and g["n_feas"] == 0 and len(g["top_idx"]) == 0
    # k larger than the feasible set
    inst3 = synth.make_instance([3, 3], seed=2, vram_cap=1e9, sla_range=(-0.05, 0.05))
    r = orc.Problem(inst3).search(inst3.sla, inst3.omega, k=64)
    g = mf.Problem(inst3).search(inst3.sla, inst3.omega, k=64)
    assert g["n_feas"] == r["n_feas"] and len(g["top_idx"]) == r["n_feas"] <= 9
    assert list(g["top_idx"]) == list(r["top_idx"])


def test_symmetric_ties(mf, orc):
    inst = synth.make_instance([9, 9], seed=11, vram_cap=1e9, symmetric=True, sla_range=(3.0, 3.0))
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=8)
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=8)
    assert list(g["top_idx"]) == list(r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_split_ranges_merge(mf):
    inst = synth.cfg1(1)
    p = mf.Problem(inst)
    full = p.search(inst.sla, inst.omega, k=16)
    cuts = [0, 1, 33_333, 33_334, 70_000, inst.space_size]
    parts = [p.search(inst.sla, inst.omega, k=16, lo=a, hi=b) for a, b in zip(cuts, cuts[1:])]
    assert sum(x["n_feas"] for x in parts) == full["n_feas"]
    assert sum(x["n_vram"] for x in parts) == full["n_vram"]
    allk = sorted([(-J, int(i)) for x in parts for J, i in zip(x["top_J"], x["top_idx"])])[:16]
    assert [i for _, i in allk] == [int(i) for i in full["top_idx"]]


def test_eval_fast_and_canonical_sampled_full_size(mf, orc):
    # sampled outputs at the full N=6 size: fast predictions within tolerance,
    # canonical predictions and J bit-identical to the oracle
    inst = synth.cfg2(0)
    rng = np.random.default_rng(0)
    idx = rng.integers(0, inst.space_size, 20_000, dtype=np.int64)
    idx[:3] = [0, inst.space_size - 1, inst.space_size // 2]
    p = mf.Problem(inst)
    fast = p.eval_fast(idx).cpu().numpy()
    can = p.eval_canonical(idx, inst.sla, inst.omega)
    ref = orc.Problem(inst).eval_list(idx.astype(np.uint64), inst.sla, inst.omega)
    rp = np.stack([ref["lat"], ref["thr"]], axis=-1)
    check_predictions(fast, rp)
    cp = can["pred"].cpu().numpy()
    assert cp.tobytes() == rp.tobytes()
    assert can["J"].cpu().numpy().tobytes() == ref["J"].tobytes()
    np.testing.assert_array_equal(can["flags"].cpu().numpy().astype(np.uint32) & 0xFFFF07,
                                  ref["flags"] & 0xFFFF07)


def test_topk_fallback_on_exact_ties(mf, orc):
    # throughput independent of the configuration: every feasible config has
    # J = N exactly, the fast list cannot separate the k-th candidate from
    # the rest, and the fallback pass gathers and certifies all of them
    inst = synth.make_instance([12, 12, 9], seed=4, vram_quantile=0.7, sla_range=(0.2, 1.0))
    for i in range(inst.n_models):
        W1, b1, W2, b2, W3, b3 = inst.model_weights(i)
        W3[1, :] = 0.0
        b3[1] = 1.0
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=5)
    assert r["n_feas"] > 64            # more tied candidates than the fast list holds
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=5)
    assert g["n_topk_collect"] > 0
    assert g["n_feas"] == r["n_feas"]
    assert list(g["top_idx"]) == list(r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_range_splits_when_certification_list_fills(mf, orc):
    inst = synth.make_instance([12, 12, 9, 9, 9], seed=5, vram_quantile=0.75,
                               sla_range=(-0.15, 0.15), top_k=16)
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=16)
    g0 = mf.Problem(inst).search(inst.sla, inst.omega, k=16)
    assert g0["n_flagged"] >= 8
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=16, worklist_cap=4)
    assert g["n_splits"] > 0, g0["n_flagged"]
    assert g["n_feas"] == r["n_feas"] and g["n_vram"] == r["n_vram"]
    assert list(g["top_idx"]) == list(r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_two_level_selection_on_long_ranges(mf, orc):
    # ranges above 2^20 configurations select the exact top-k in two levels
    # (a grid of partial lists, then one merge): a full search, and exact
    # ties that force the collect pass through the same path
    inst = synth.make_instance([17, 16, 16, 16, 16], seed=6, vram_quantile=0.6, sla_range=(0.3, 1.2))
    assert inst.space_size > 2 ** 20
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=16)
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=16)
    assert g["n_vram"] == r["n_vram"] and g["n_feas"] == r["n_feas"]
    assert list(g["top_idx"]) == list(r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()
    for i in range(inst.n_models):
        W1, b1, W2, b2, W3, b3 = inst.model_weights(i)
        W3[1, :] = 0.0
        b3[1] = 1.0
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=7)
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=7)
    assert g["n_topk_collect"] > 0
    assert g["n_feas"] == r["n_feas"]
    assert list(g["top_idx"]) == list(r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_search_argument_errors(mf, orc):
    # every invalid argument is refused before any launch, with the status the
    # header documents, and the problem still searches correctly afterwards
    import ctypes as C
    import torch
    inst = synth.cfg1(1)
    p = mf.Problem(inst)
    d_sla = torch.as_tensor(inst.sla, dtype=torch.float32, device="cuda")
    d_om = torch.as_tensor(inst.omega, dtype=torch.float32, device="cuda")

    def args(**over):
        a = dict(lo=0, hi=inst.space_size, top_k=4, flags=0, d_sla=d_sla.data_ptr(), d_omega=d_om.data_ptr(),
                 d_mask=None, d_pred=None)
        a.update(over)
        return mf.SearchArgs(a["lo"], a["hi"], a["top_k"], a["flags"], a["d_sla"], a["d_omega"], a["d_mask"],
                             a["d_pred"], mf.objective_args(None, inst.n_models))

    def size(a):
        n = C.c_size_t()
        return mf.lib.mf_workspace_size(p.handle, C.byref(a), C.byref(n)), n.value

    st, need = size(args())
    assert st == mf.MF_OK and need > 0
    ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
    assert ws.data_ptr() % 256 == 0
    res = mf.Result()

    def search(a, ptr=ws.data_ptr(), nbytes=need):
        return mf.lib.mf_search(p.handle, C.byref(a), C.c_void_p(ptr), C.c_size_t(nbytes),
                                C.c_void_p(torch.cuda.current_stream().cuda_stream), C.byref(res))

    cases = [
        (args(top_k=0), mf.MF_EINVAL),
        (args(top_k=65), mf.MF_EINVAL),
        (args(lo=10, hi=9), mf.MF_EINVAL),
        (args(hi=inst.space_size + 1), mf.MF_EOVERFLOW),
        (args(d_sla=None), mf.MF_EINVAL),
        (args(d_omega=None), mf.MF_EINVAL),
        (args(flags=1 << 7), mf.MF_EINVAL),
        (args(flags=mf.MF_DUMP), mf.MF_EINVAL),          # dump without its buffers
    ]
    for a, want in cases:
        assert size(a)[0] == want
        assert search(a) == want
    assert search(args(), nbytes=need - 1) == mf.MF_ENOMEM
    assert search(args(), ptr=ws.data_ptr() + 128) == mf.MF_EINVAL   # workspace not 256-byte aligned
    assert search(args(), ptr=0) == mf.MF_EINVAL
    assert mf.lib.mf_search(p.handle, C.byref(args()), C.c_void_p(ws.data_ptr()), C.c_size_t(need), None,
                            None) == mf.MF_EINVAL
    assert search(args()) == mf.MF_OK
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=4)
    assert res.n_feas == r["n_feas"] and res.n_vram == r["n_vram"]
    assert [int(x) for x in res.top_idx[:res.n_top]] == list(r["top_idx"])
    assert all(x == 2 ** 64 - 1 for x in res.top_idx[res.n_top:])
    p.close()


def test_repeated_runs_are_bit_identical(mf):
    # the same search twice, and once more after other work on the problem:
    # counts, top-k, masks and fast-path predictions identical byte for byte
    inst = synth.cfg2(2)
    p = mf.Problem(inst)
    lo, hi = 12_345_678, 12_345_678 + 700_001
    a = p.search(inst.sla, inst.omega, k=16, lo=lo, hi=hi, dump=True)
    b = p.search(inst.sla, inst.omega, k=16, lo=lo, hi=hi, dump=True)
    p.search(inst.sla * 1.1, inst.omega, k=64, lo=0, hi=3_000_000)
    c = p.search(inst.sla, inst.omega, k=16, lo=lo, hi=hi, dump=True)
    for x in (b, c):
        for key in ("n_eval", "n_vram", "n_feas", "n_flagged"):
            assert x[key] == a[key]
        assert x["top_idx"].tobytes() == a["top_idx"].tobytes()
        assert x["top_J"].tobytes() == a["top_J"].tobytes()
        assert x["mask"].cpu().numpy().tobytes() == a["mask"].cpu().numpy().tobytes()
        assert x["pred"].cpu().numpy().tobytes() == a["pred"].cpu().numpy().tobytes()
    p.close()
