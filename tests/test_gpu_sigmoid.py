"""GPU parity with the surrogates' sigmoid output (Section III-B: the
predictor ends in a sigmoid) against the CPU oracle, through the C ABI: the
fp32 and bf16 searches, the full utility of Eq. 3, the fixed observed state,
the static search, the GA, and the canonical evaluation.

Bars as elsewhere: masks, counts, top-k and canonical J bit-exact (the
canonical sigmoid is one algorithm on both sides, so canonical predictions
agree bit for bit); fast predictions within 1e-5 (fp32) or 2e-2 (bf16).
"""
import numpy as np
import pytest

from paper_2609_02109_amd import synth
from test_gpu_search import check_predictions

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_02109_amd import mf as mfmod
    return mfmod


def sig_instance(orc, n_options, L, A, H, seed, dtype="f32", q=0.7, vram_quantile=0.8):
    """A sigmoid-output instance with each model's latency bound at the q-th
    quantile of its oracle latencies over a sample of configurations."""
    inst = synth.make_instance(n_options, L, A, H, H, seed=seed, vram_quantile=vram_quantile, dtype=dtype,
                               act="sigmoid", sla_range=(0.5, 0.5))
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, inst.space_size, 2_000).astype(np.uint64)
    lat = orc.Problem(inst).eval_list(idx, np.full(inst.n_models, np.inf, np.float32), inst.omega)["lat"]
    inst.sla = np.quantile(lat, q, axis=0).astype(np.float32)
    return inst


def parity(mf, orc, inst, lo, hi, k, tol, ob=None, state=None):
    print(f"[sigmoid] {inst.name} seed={inst.seed} {inst.dtype} range=[{lo},{hi}) k={k} eq3={ob is not None} "
          f"fixed={state is not None}", flush=True)
    g = mf.Problem(inst, variants=ob).search(inst.sla, inst.omega, k=k, lo=lo, hi=hi, dump=True, objective=ob,
                                             state=state)
    r = orc.Problem(inst, ob, state=state).search(inst.sla, inst.omega, k=k, lo=lo, hi=hi, dump=True)
    assert g["n_vram"] == r["n_vram"] and g["n_feas"] == r["n_feas"]
    gm = g["mask"].cpu().numpy().astype(np.uint32)
    np.testing.assert_array_equal(gm & 7, r["flags"] & 7)
    np.testing.assert_array_equal(g["top_idx"], r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()
    check_predictions(g["pred"].cpu().numpy(), r["pred"], tol=tol)
    return g, r


def test_sigmoid_fp32_full_spaces(mf, orc):
    inst = sig_instance(orc, [12, 12, 9, 9, 9], 8, 4, 32, seed=1)
    g, r = parity(mf, orc, inst, 0, inst.space_size, 16, 1e-5)
    assert 0 < r["n_feas"] < r["n_vram"]
    inst2 = sig_instance(orc, [6, 6], 8, 4, 32, seed=2, q=0.5)
    parity(mf, orc, inst2, 0, inst2.space_size, 1, 1e-5)


def test_sigmoid_fp32_n6_ranges(mf, orc):
    inst = sig_instance(orc, [24] * 6, 16, 6, 64, seed=0, q=0.8, vram_quantile=0.9)
    n = inst.space_size
    parity(mf, orc, inst, 0, 120_000, 4, 1e-5)
    parity(mf, orc, inst, n - 70_001, n, 8, 1e-5)


def test_sigmoid_bf16(mf, orc):
    inst = sig_instance(orc, [7, 9, 3, 5], 12, 8, 128, seed=9, dtype="bf16")
    parity(mf, orc, inst, 0, inst.space_size, 9, 2e-2)
    inst8 = sig_instance(orc, [16] * 8, 32, 8, 256, seed=1, dtype="bf16", q=0.85, vram_quantile=0.95)
    parity(mf, orc, inst8, 2 ** 31 - 4_000, 2 ** 31 + 4_000, 64, 2e-2)


def test_sigmoid_eq3_and_fixed_state(mf, orc):
    inst = sig_instance(orc, [12, 12, 9, 9, 9], 8, 4, 32, seed=4)
    ob = synth.make_objective(inst, 4, tau_range=(0.2, 0.4))
    g, r = parity(mf, orc, inst, 0, inst.space_size, 16, 1e-5, ob=ob)
    assert r["n_feas"] > 0
    st = synth.make_state(inst, 4)
    parity(mf, orc, inst, 0, inst.space_size, 16, 1e-5, ob=ob, state=st)
    bf = sig_instance(orc, [6, 5, 4], 8, 4, 64, seed=5, dtype="bf16")
    obb = synth.make_objective(bf, 5)
    parity(mf, orc, bf, 0, bf.space_size, 5, 2e-2, ob=obb)


def test_sigmoid_static_and_ga(mf, orc):
    inst = sig_instance(orc, [12, 12, 9, 9, 9], 8, 4, 32, seed=6)
    ob = synth.make_objective(inst, 6)
    sc = synth.make_scenarios(inst, 1, 4, seed=6, latency_bounds=True)
    g = mf.Problem(inst, variants=ob).search_static(sc.states[0], sc.sla[0], sc.omega[0], k=8, objective=ob)
    r = orc.static_search(inst, ob, sc.states[0], sc.sla[0], sc.omega[0], k=8)
    assert g["n_feas"] == r["n_feas"] and list(g["top_idx"]) == list(r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()
    gs = synth.ga_scenarios(5, 3, seed=6)
    gsla = np.broadcast_to(inst.sla, gs.sla.shape).copy()
    ga = mf.Problem(inst, variants=ob).ga(gsla, gs.omega, pop=64, gens=6, seed=4, final_pop=True, objective=ob)
    gr = orc.Problem(inst, ob).ga(gsla, gs.omega, pop=64, gens=6, seed=4, final_pop=True)
    np.testing.assert_array_equal(ga["best_idx"], gr["best_idx"])
    assert ga["best_J"].tobytes() == gr["best_J"].tobytes()
    np.testing.assert_array_equal(ga["final_pop"].cpu().numpy().astype(np.uint64), gr["final_pop"])


def test_sigmoid_canonical_evaluation_bitwise(mf, orc):
    for inst in (sig_instance(orc, [12, 12, 9, 9, 9], 8, 4, 32, seed=7),
                 sig_instance(orc, [7, 9, 3, 5], 12, 8, 128, seed=7, dtype="bf16")):
        rng = np.random.default_rng(7)
        idx = rng.integers(0, inst.space_size, 3_000).astype(np.int64)
        can = mf.Problem(inst).eval_canonical(idx, inst.sla, inst.omega)
        ref = orc.Problem(inst).eval_list(idx.astype(np.uint64), inst.sla, inst.omega)
        rp = np.stack([ref["lat"], ref["thr"]], axis=-1)
        assert can["pred"].cpu().numpy().tobytes() == rp.tobytes()
        assert can["J"].cpu().numpy().tobytes() == ref["J"].tobytes()
        fast = mf.Problem(inst).eval_fast(idx).cpu().numpy()
        check_predictions(fast, rp, tol=1e-5 if inst.dtype == "f32" else 2e-2)


def test_sigmoid_rejects_unknown_activation(mf):
    inst = synth.cfg0(0)
    p = mf.Problem(inst)
    d = p.desc
    d.output_act = 7
    import ctypes as C
    h = C.c_void_p()
    import torch
    feats = torch.as_tensor(inst.features, device="cuda")
    w = torch.as_tensor(inst.weights, device="cuda")
    tables = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    st = mf.lib.mf_problem_create(C.byref(d), C.c_void_p(feats.data_ptr()), C.c_void_p(w.data_ptr()),
                                  C.c_void_p(tables.data_ptr()), tables.numel(), None, C.byref(h))
    assert st == mf.MF_EINVAL
