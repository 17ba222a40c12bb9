"""GPU parity of the search under the full utility (Section II, Eq. 3) with
the throughput floor, against the CPU oracle, through the C ABI.

Bars: VRAM / service / feasible masks, n_vram, n_feas, top-k indices and
canonical J bit-exact; fast predictions within the fp32 (1e-5) or bf16 (2e-2)
tolerance.
"""
from dataclasses import replace

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


def eq3_parity(mf, orc, inst, ob, lo, hi, k, tol=1e-5):
    print(f"[eq3] {inst.name} seed={inst.seed} range=[{lo},{hi}) k={k}", flush=True)
    p = mf.Problem(inst, variants=ob)
    g = p.search(inst.sla, inst.omega, k=k, lo=lo, hi=hi, dump=True, objective=ob)
    r = orc.Problem(inst, ob).search(inst.sla, inst.omega, k=k, lo=lo, hi=hi, dump=True)
    assert g["n_eval"] == hi - lo
    assert g["n_vram"] == r["n_vram"]
    assert g["n_feas"] == r["n_feas"]
    gm = g["mask"].cpu().numpy().astype(np.uint32)
    rf = r["flags"]
    np.testing.assert_array_equal(gm & 1, rf & 1)
    np.testing.assert_array_equal((gm >> 1) & 1, (rf >> 1) & 1)
    np.testing.assert_array_equal((gm >> 2) & 1, (rf >> 2) & 1)
    np.testing.assert_array_equal(g["top_idx"], r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()
    check_predictions(g["pred"].cpu().numpy(), r["pred"], tol=tol)
    p.close()
    return g, r


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_eq3_n5_full(mf, orc, seed):
    inst = synth.cfg1(seed)
    g, r = eq3_parity(mf, orc, inst, synth.make_objective(inst, seed), 0, inst.space_size, 16)
    assert 0 < r["n_feas"] < r["n_vram"]


def test_eq3_n2_full(mf, orc):
    inst = synth.cfg0(1)
    eq3_parity(mf, orc, inst, synth.make_objective(inst, 3), 0, inst.space_size, 1)


def test_eq3_tight_floors(mf, orc):
    # floors drawn inside the normalised throughput's range, so many floor
    # decisions sit close to their bound and go to the canonical pass
    inst = synth.make_instance([12, 12, 9, 9, 9], seed=8, vram_quantile=0.8, sla_range=(1.0, 2.0), top_k=16)
    ob = synth.make_objective(inst, 8, tau_range=(0.45, 0.55))
    g, r = eq3_parity(mf, orc, inst, ob, 0, inst.space_size, 16)
    assert g["n_flagged"] > 0 and r["n_feas"] > 0


def test_eq3_n6_ragged_ranges(mf, orc):
    inst = synth.cfg2(0)
    ob = synth.make_objective(inst, 0)
    n = inst.space_size
    eq3_parity(mf, orc, inst, ob, 0, 150_000, 4)
    eq3_parity(mf, orc, inst, ob, n - 50_001, n, 8)


def test_eq3_bf16(mf, orc):
    inst = synth.make_instance([7, 9, 3, 5], 12, 8, 128, 128, seed=9, vram_quantile=0.7, sla_range=(0.0, 1.0),
                               dtype="bf16")
    eq3_parity(mf, orc, inst, synth.make_objective(inst, 9), 0, inst.space_size, 9, tol=2e-2)
    inst8 = synth.cfg4(1)
    eq3_parity(mf, orc, inst8, synth.make_objective(inst8, 1), 2 ** 31 - 6_000, 2 ** 31 + 6_000, 64, tol=2e-2)


def test_eq3_linear_special_case_matches_linear_search(mf):
    for inst in (synth.cfg1(2), synth.make_instance([6, 5, 4], 8, 4, 64, 64, seed=3, vram_quantile=0.6,
                                                    sla_range=(-0.2, 0.8), dtype="bf16")):
        p = mf.Problem(inst, variants=synth.linear_objective(inst))
        a = p.search(inst.sla, inst.omega, k=16)
        b = p.search(inst.sla, inst.omega, k=16, objective=synth.linear_objective(inst))
        assert a["n_feas"] == b["n_feas"] and a["n_vram"] == b["n_vram"]
        assert list(a["top_idx"]) == list(b["top_idx"])
        assert a["top_J"].tobytes() == b["top_J"].tobytes()


def test_eq3_reload_ties_use_the_fallback(mf, orc):
    # Q = 0, no penalty, no floor: J = -alpha sum_i c_i eta_i takes a handful
    # of values, each shared by thousands of configurations; with no previous
    # deployment as well, J = 0 everywhere and the exact top-k needs the
    # fallback pass (every tied configuration with the lowest indices)
    inst = synth.make_instance([12, 12, 9, 9, 9], seed=4, vram_quantile=0.9, sla_range=(1e9, 1e9))
    ob = replace(synth.make_objective(inst, 4), quality=np.zeros((5, synth.MAX_VARIANTS), np.float32),
                 tau=np.full(5, -np.inf, np.float32), beta=0.0)
    for o, must_collect in ((ob, False), (replace(ob, prev_variant=np.full(5, -1, np.int32)), True)):
        r = orc.Problem(inst, o).search(inst.sla, inst.omega, k=64)
        g = mf.Problem(inst, variants=o).search(inst.sla, inst.omega, k=64, objective=o)
        if must_collect:
            assert g["n_topk_collect"] > 0
        assert g["n_feas"] == r["n_feas"]
        assert list(g["top_idx"]) == list(r["top_idx"])
        assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_eq3_argument_validation(mf):
    inst = synth.cfg1(0)
    ob = synth.make_objective(inst, 0)
    plain = mf.Problem(inst)
    with pytest.raises(mf.MfError) as e:
        plain.search(inst.sla, inst.omega, k=1, objective=ob)   # no variants at creation
    assert e.value.status == mf.MF_EINVAL
    p = mf.Problem(inst, variants=ob)
    for bad in (replace(ob, prev_variant=np.array([0, 0, 5, 0, 0], np.int32)),
                replace(ob, tau=np.array([0.3, np.nan, 0.3, 0.3, 0.3], np.float32)),
                replace(ob, tau=np.array([0.3, np.inf, 0.3, 0.3, 0.3], np.float32)),
                replace(ob, beta=-1.0), replace(ob, alpha=np.inf)):
        with pytest.raises(mf.MfError) as e:
            p.search(inst.sla, inst.omega, k=1, objective=bad)
        assert e.value.status == mf.MF_EINVAL
    for bad in (replace(ob, fmax=ob.fmin.copy()), replace(ob, n_variants=np.array([2, 2, 5, 3, 3], np.int32)),
                replace(ob, variant=np.full_like(ob.variant, 3))):
        with pytest.raises(mf.MfError) as e:
            mf.Problem(inst, variants=bad)
        assert e.value.status == mf.MF_EINVAL
