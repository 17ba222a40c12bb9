"""Pins for the oracle of the scheduling protocol (Section IV-C, Table II).

  * exhaustive decisions are the brute-force argmax of each step's utility
    under the scheduler's own previous deployment (numpy over the step's full
    dump, not the oracle's top-k);
  * no GA decision beats the exhaustive optimum of its own step and previous
    deployment;
  * the static choices are ordered by access: S(static_full) >=
    S(budget 5000) >= S(budget 500) (the 500 samples are a prefix of the
    5000);
  * with one step and no previous deployment, static_full and exhaustive
    decide the same configuration;
  * Random's decisions meet the VRAM cap whenever one of its candidates does;
  * the metric formulas on a hand-made run.
"""
from dataclasses import replace

import numpy as np
import pytest

from paper_2609_02109_amd import synth
from paper_2609_02109_amd.protocol import ProtocolParams, scheduler_names


@pytest.fixture(scope="module")
def small_run(orc):
    import oracle.protocol as op
    inst = synth.cfg1(1)
    ob = synth.make_objective(inst, 1)
    sc = synth.make_scenarios(inst, 2, 4, seed=1)
    dr = synth.protocol_draws(inst, 2, 4, seed=1)
    P = ProtocolParams(ga_pop=32, ga_gens=6)
    return inst, ob, sc, dr, P, op.run(inst, ob, sc, dr, P, scheduler_names(P))


def prev_of(inst, ob, idx):
    d = np.array(np.unravel_index(int(idx), tuple(int(k) for k in inst.n_options)))
    return ob.variant[inst.option_offsets + d].astype(np.int32)


def test_exhaustive_is_the_brute_force_argmax(orc, small_run):
    inst, ob, sc, dr, P, r = small_run
    for s in range(2):
        prev = ob.prev_variant
        for t in range(4):
            ob_t = replace(ob, prev_variant=prev)
            d = orc.Problem(inst, ob_t, state=sc.states[s, t]).search(sc.sla[s, t], sc.omega[s, t], dump=True)
            J = d["J"]
            best = int(np.lexsort((np.arange(len(J)), -J))[0])
            assert np.isfinite(J[best])
            assert int(r["exhaustive"]["idx"][s, t]) == best
            assert r["exhaustive"]["J"][s, t] == J[best]
            prev = prev_of(inst, ob, best)


def test_ga_never_beats_its_steps_optimum(orc, small_run):
    inst, ob, sc, dr, P, r = small_run
    for s in range(2):
        prev = ob.prev_variant
        for t in range(4):
            ob_t = replace(ob, prev_variant=prev)
            top = orc.Problem(inst, ob_t, state=sc.states[s, t]).search(sc.sla[s, t], sc.omega[s, t], k=1)
            assert r["ga"]["J"][s, t] <= top["top_J"][0]
            prev = prev_of(inst, ob, r["ga"]["idx"][s, t])


def test_static_choices_are_ordered_by_access(orc, small_run):
    inst, ob, sc, dr, P, r = small_run
    for s in range(2):
        S = {}
        for name in ("static_full", "static_budget_5000", "static_budget_500"):
            idx = np.array([r[name]["idx"][s, 0]], np.uint64)
            _, _, S[name] = orc.static_eval(inst, ob, sc.states[s], sc.sla[s], sc.omega[s], idx)
            assert (r[name]["idx"][s] == idx[0]).all()
        assert S["static_full"][0] >= S["static_budget_5000"][0] >= S["static_budget_500"][0]


def test_one_step_static_full_is_exhaustive(orc):
    import oracle.protocol as op
    inst = synth.cfg1(2)
    ob = replace(synth.make_objective(inst, 2), prev_variant=np.full(inst.n_models, -1, np.int32))
    sc = synth.make_scenarios(inst, 3, 1, seed=2)
    dr = synth.protocol_draws(inst, 3, 1, seed=2)
    P = ProtocolParams(budgets=(50,), ga_pop=8, ga_gens=1)
    r = op.run(inst, ob, sc, dr, P, ["exhaustive", "static_full"])
    np.testing.assert_array_equal(r["exhaustive"]["idx"], r["static_full"]["idx"])
    assert r["exhaustive"]["J"].tobytes() == r["static_full"]["J"].tobytes()


def test_random_meets_the_vram_cap(orc, small_run):
    inst, ob, sc, dr, P, r = small_run
    for s in range(2):
        for t in range(4):
            cand = dr.random[s, t]
            fl = orc.Problem(inst, ob, state=sc.states[s, t]).eval_list(cand, sc.sla[s, t], sc.omega[s, t],
                                                                      raw=True)["flags"]
            within = cand[(fl & orc.FLAG_VRAM) != 0]
            assert int(r["random"]["idx"][s, t]) == int(within[0] if len(within) else cand[0])


def test_metric_formulas():
    import oracle.protocol as op
    run = {"exhaustive": dict(J=np.array([[2.0, 4.0], [1.0, 1.0]]), ok=np.ones((2, 2), bool)),
           "x": dict(J=np.array([[1.5, 3.0], [1.0, 0.5]]), ok=np.array([[True, False], [True, True]]))}
    t = op.table([run])
    assert t["exhaustive"] == dict(mean_J=2.0, avg_gap=0.0, worst_gap=0.0, sla_pct=0.0)
    # scenario gaps: (3 - 2.25) / 3 = 25 %, (1 - 0.75) / 1 = 25 %
    assert t["x"]["mean_J"] == 1.5 and t["x"]["avg_gap"] == 25.0 and t["x"]["worst_gap"] == 25.0
    assert t["x"]["sla_pct"] == 25.0
