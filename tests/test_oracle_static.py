"""Pins for the oracle's static (multi-step) evaluation: one configuration held
over T decision steps, S = sum_t J_t in step order (the static schedulers of
Section IV-C, Table II).

  * T = 1 is the single-step fixed-state search (itself pinned in
    test_oracle_fixed_state.py and test_oracle_objective.py);
  * two identical steps with no reload give S = 2 J exactly (doubling is
    exact), so the same ranking as one step;
  * the feasible set over T steps is the intersection of the steps' feasible
    sets (VRAM once, every step's floors and bounds);
  * the reload term enters at step 0 only: with only alpha non-zero, S takes
    the closed-form values of the reload histogram of step 0;
  * the raw utility of a configuration that breaks a floor equals the
    feasible value of the same configuration under a floor it meets.
"""
from dataclasses import replace

import numpy as np

from paper_2609_02109_amd import synth


def steps_of(sc, s):
    return sc.states[s], sc.sla[s], sc.omega[s]


def test_static_one_step_is_the_fixed_state_search(orc):
    inst = synth.cfg1(0)
    ob = synth.make_objective(inst, 0)
    sc = synth.make_scenarios(inst, 2, 1, seed=0)
    for s in range(2):
        st, sla, om = steps_of(sc, s)
        r1 = orc.static_search(inst, ob, st, sla, om, k=16)
        r0 = orc.Problem(inst, ob, state=st[0]).search(sla[0], om[0], k=16)
        assert r1["n_feas"] == r0["n_feas"] and r1["n_vram"] == r0["n_vram"]
        assert list(r1["top_idx"]) == list(r0["top_idx"])
        assert r1["top_J"].tobytes() == r0["top_J"].tobytes()


def test_static_two_identical_steps_double_exactly(orc):
    inst = synth.cfg1(1)
    ob = replace(synth.make_objective(inst, 1), prev_variant=np.full(inst.n_models, -1, np.int32))
    st = np.stack([synth.make_state(inst, 1)] * 2)
    sla = np.stack([inst.sla] * 2)
    om = np.stack([inst.omega] * 2)
    r2 = orc.static_search(inst, ob, st, sla, om, k=8)
    r1 = orc.static_search(inst, ob, st[:1], sla[:1], om[:1], k=8)
    assert r2["n_feas"] == r1["n_feas"]
    assert list(r2["top_idx"]) == list(r1["top_idx"])
    assert (r2["top_J"] == 2.0 * r1["top_J"]).all()
    feas = (r2["flags"] & orc.FLAG_FEAS) != 0
    assert (r2["S"][feas] == 2.0 * r1["S"][feas]).all()


def test_static_feasible_set_is_the_intersection(orc):
    inst = synth.cfg1(2)
    ob = synth.make_objective(inst, 2, tau_range=(0.3, 0.5))
    sc = synth.make_scenarios(inst, 1, 5, seed=2, latency_bounds=True)
    st, sla, om = steps_of(sc, 0)
    r = orc.static_search(inst, ob, st, sla, om, k=4)
    per = [orc.Problem(inst, ob, state=st[t]).search(sla[t], om[t], dump=True)["flags"] for t in range(5)]
    inter = np.logical_and.reduce([(f & orc.FLAG_FEAS) != 0 for f in per])
    assert r["n_feas"] == int(inter.sum())
    assert 0 < r["n_feas"] < min(int(((f & orc.FLAG_FEAS) != 0).sum()) for f in per)
    assert r["n_vram"] == int(((per[0] & orc.FLAG_VRAM) != 0).sum())


def test_static_reload_only_at_step_zero(orc):
    # Q = 0, no penalty, no floor, alpha = 1, c_i = 2^i: every step after the
    # first adds exactly 0, so S = J_0 = -(sum of 2^i over changed models)
    inst = synth.make_instance([6, 4, 9], seed=2, vram_cap=1e9, sla_range=(1e9, 1e9))
    ob = synth.make_objective(inst, seed=5)
    ob = replace(ob, quality=np.zeros_like(ob.quality), reload_cost=np.array([1, 2, 4], np.float32),
                 tau=np.full(3, -np.inf, np.float32), alpha=1.0, beta=0.0)
    sc = synth.make_scenarios(inst, 1, 4, seed=3)
    st, sla, om = steps_of(sc, 0)
    r = orc.static_search(inst, ob, st, sla, om, k=1)
    offs = np.concatenate([[0], np.cumsum(inst.n_options)])
    digits = np.array(np.unravel_index(np.arange(inst.space_size), tuple(int(k) for k in inst.n_options))).T
    changed = np.stack([ob.variant[offs[i] + digits[:, i]] != ob.prev_variant[i] for i in range(3)], axis=1)
    want = -(changed * np.array([1.0, 2.0, 4.0])).sum(axis=1)
    assert (r["S"] == want).all()
    assert (r["J"][:, 1:] == 0.0).all()


def test_static_raw_utility_of_a_floor_violation(orc):
    inst = synth.cfg1(0)
    ob = synth.make_objective(inst, 0, tau_range=(0.45, 0.55))
    st = synth.make_state(inst, 0)[None, :]
    sla = np.full((1, inst.n_models), np.inf, np.float32)
    om = inst.omega[None, :]
    idx = np.arange(0, inst.space_size, 97, dtype=np.uint64)
    J, F, S = orc.static_eval(inst, ob, st, sla, om, idx)
    bad = (F[:, 0] & orc.FLAG_SLA) == 0
    assert bad.any() and (~bad).any()
    # the same configurations under floors they meet: the value moves only
    # by the penalty terms, which vanish with beta = 0 and tau = -inf
    lo = replace(ob, tau=np.full(inst.n_models, -np.inf, np.float32), beta=0.0)
    J0, F0, _ = orc.static_eval(inst, replace(ob, beta=0.0), st, sla, om, idx)
    J1, F1, _ = orc.static_eval(inst, lo, st, sla, om, idx)
    assert np.isfinite(J0).all() and (J0 == J1).all()
    assert ((F1[:, 0] & orc.FLAG_SLA) != 0).all()
