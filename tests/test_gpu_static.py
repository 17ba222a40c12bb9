"""GPU parity of the static (multi-step) search and evaluation against the CPU
oracle's step-by-step composition, through the C ABI.

Bars: VRAM / service / feasible masks, n_vram, n_feas, top-k indices and S
(the step-order sum of canonical utilities) bit-exact; per-step utilities
and flags of index lists bit-exact.
"""
from dataclasses import replace

import numpy as np
import pytest

from paper_2609_02109_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_02109_amd import mf as mfmod
    return mfmod


def static_parity(mf, orc, inst, ob, st, sla, om, k, lo=0, hi=None):
    hi = inst.space_size if hi is None else hi
    print(f"[static] {inst.name} seed={inst.seed} T={len(st)} range=[{lo},{hi}) k={k} eq3={ob is not None}",
          flush=True)
    g = mf.Problem(inst, variants=ob).search_static(st, sla, om, k=k, lo=lo, hi=hi, objective=ob, dump=True)
    r = orc.static_search(inst, ob, st, sla, om, k=k, lo=lo, hi=hi)
    assert g["n_eval"] == hi - lo
    assert g["n_vram"] == r["n_vram"] and g["n_feas"] == r["n_feas"]
    np.testing.assert_array_equal(g["mask"].cpu().numpy().astype(np.uint32), r["flags"])
    np.testing.assert_array_equal(g["top_idx"], r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()
    return g, r


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_static_n5_eq3_full(mf, orc, seed):
    inst = synth.cfg1(seed)
    sc = synth.make_scenarios(inst, 1, 12, seed=seed)
    g, r = static_parity(mf, orc, inst, synth.make_objective(inst, seed), sc.states[0], sc.sla[0], sc.omega[0], 16)
    assert r["n_feas"] > 16


def test_static_n5_linear_with_latency_bounds(mf, orc):
    inst = synth.cfg1(1)
    sc = synth.make_scenarios(inst, 2, 5, seed=4, latency_bounds=True)
    for s in range(2):
        static_parity(mf, orc, inst, None, sc.states[s], sc.sla[s], sc.omega[s], 8)


def test_static_n6_ranges(mf, orc):
    inst = synth.cfg2(0)
    ob = synth.make_objective(inst, 0)
    sc = synth.make_scenarios(inst, 1, 4, seed=5)
    n = inst.space_size
    static_parity(mf, orc, inst, ob, sc.states[0], sc.sla[0], sc.omega[0], 8, 0, 60_000)
    static_parity(mf, orc, inst, ob, sc.states[0], sc.sla[0], sc.omega[0], 8, n - 30_001, n)


def test_static_bf16_and_many_models(mf, orc):
    inst = synth.make_instance([7, 9, 3, 5], 12, 8, 128, 128, seed=9, vram_quantile=0.7, dtype="bf16")
    sc = synth.make_scenarios(inst, 1, 3, seed=9)
    static_parity(mf, orc, inst, synth.make_objective(inst, 9), sc.states[0], sc.sla[0], sc.omega[0], 9)
    inst16 = synth.make_instance([2] * 16, 8, 4, 32, 32, seed=3, vram_quantile=0.6)
    sc = synth.make_scenarios(inst16, 1, 6, seed=3, latency_bounds=True)
    static_parity(mf, orc, inst16, None, sc.states[0], sc.sla[0], sc.omega[0], 5)


def test_static_one_step_equals_fixed_state_search(mf):
    inst = synth.cfg2(1)
    ob = synth.make_objective(inst, 1)
    st = synth.make_state(inst, 1)
    p = mf.Problem(inst, variants=ob)
    a = p.search(inst.sla, inst.omega, k=16, objective=ob, state=st)
    b = p.search_static(st[None, :], inst.sla[None, :], inst.omega[None, :], k=16, objective=ob)
    assert a["n_feas"] == b["n_feas"] and a["n_vram"] == b["n_vram"]
    assert list(a["top_idx"]) == list(b["top_idx"])
    assert a["top_J"].tobytes() == b["top_J"].tobytes()


def test_static_eval_lists(mf, orc):
    inst = synth.cfg1(2)
    ob = synth.make_objective(inst, 2, tau_range=(0.4, 0.55))
    sc = synth.make_scenarios(inst, 1, 7, seed=2)
    rng = np.random.default_rng(3)
    idx = rng.integers(0, inst.space_size, 5_000).astype(np.uint64)
    idx[:2] = [0, inst.space_size - 1]
    g = mf.Problem(inst, variants=ob).eval_static(idx, sc.states[0], sc.sla[0], sc.omega[0], objective=ob)
    J, F, S = orc.static_eval(inst, ob, sc.states[0], sc.sla[0], sc.omega[0], idx)
    assert g["J"].tobytes() == J.tobytes()
    assert g["S"].tobytes() == S.tobytes()
    np.testing.assert_array_equal(g["flags"], F & 3)
    assert ((F & 2) == 0).any() and ((F & 2) != 0).any()
    # one step with the previous decision as the previous deployment: the
    # utility a dynamic schedule records for that step
    prev = replace(ob, prev_variant=ob.variant[inst.option_offsets + np.array([3, 1, 4, 1, 5])].astype(np.int32))
    g1 = mf.Problem(inst, variants=ob).eval_static(idx, sc.states[0][2:3], sc.sla[0][2:3], sc.omega[0][2:3],
                                                   objective=prev)
    r1 = orc.Problem(inst, prev, state=sc.states[0][2]).eval_list(idx, sc.sla[0][2], sc.omega[0][2], raw=True)
    assert g1["J"][:, 0].tobytes() == r1["J"].tobytes()


def test_static_argument_validation(mf):
    inst = synth.cfg1(0)
    sc = synth.make_scenarios(inst, 1, 3, seed=0)
    p = mf.Problem(inst)
    for bad_T in (0, 33):
        st = np.zeros((bad_T, inst.n_agg), np.float32)
        with pytest.raises((mf.MfError, ValueError)):
            p.search_static(st, np.zeros((bad_T, inst.n_models)), np.ones((bad_T, inst.n_models)), k=1)
    st = sc.states[0].copy()
    st[1, 0] = np.nan
    with pytest.raises(mf.MfError) as e:
        p.search_static(st, sc.sla[0], sc.omega[0], k=1)
    assert e.value.status == mf.MF_EINVAL
    big = synth.make_instance([255] * 8, 8, 4, 32, 32, seed=1, vram_quantile=0.5)
    sc16 = synth.make_scenarios(big, 1, 32, seed=1)
    with pytest.raises(mf.MfError) as e:
        mf.Problem(big).search_static(sc16.states[0], sc16.sla[0], sc16.omega[0], k=1)
    assert e.value.status == mf.MF_EUNSUPPORTED
