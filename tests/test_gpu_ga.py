"""GPU GA (mf_ga_run) against the oracle's GA replay.

Fitness is the canonical J on both sides and every random draw comes from the
same counter-based Philox stream, so the whole trajectory is reproduced: the
best individual per scenario and the final population must be identical.
"""
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


def run_both(mf, orc, inst, sla, omega, **kw):
    print(f"[ga] {inst.name} S={len(sla)} {kw}", flush=True)
    g = mf.Problem(inst).ga(sla, omega, final_pop=True, **kw)
    r = orc.Problem(inst).ga(sla, omega, final_pop=True, **kw)
    np.testing.assert_array_equal(g["best_idx"], r["best_idx"])
    assert g["best_J"].tobytes() == r["best_J"].tobytes()
    np.testing.assert_array_equal(g["final_pop"].cpu().numpy().astype(np.uint64), r["final_pop"])
    return g, r


def test_ga_n5_subset_full_length(mf, orc):
    inst, sc, gp = synth.cfg3(0)
    run_both(mf, orc, inst, sc.sla[:8], sc.omega[:8], pop=gp.pop, gens=gp.gens, tourn_k=gp.tourn_k,
             p_cx=gp.p_cx, p_swap=gp.p_swap, p_mut=gp.p_mut, seed=gp.seed)


def test_ga_n5_all_scenarios(mf, orc):
    inst, sc, gp = synth.cfg3(1)
    g, r = run_both(mf, orc, inst, sc.sla, sc.omega, pop=gp.pop, gens=gp.gens, seed=gp.seed)
    # the GA never beats the exhaustive optimum of its scenario
    p = mf.Problem(inst)
    for s in range(0, 64, 9):
        ex = p.search(sc.sla[s], sc.omega[s], k=1)
        assert g["best_J"][s] <= ex["top_J"][0]


@pytest.mark.parametrize("kw", [dict(pop=64, gens=7, tourn_k=1, p_cx=1.0, p_mut=0.3),
                                dict(pop=130, gens=3, tourn_k=8, p_cx=0.0, p_mut=0.0),
                                dict(pop=4, gens=2, tourn_k=2)])
def test_ga_operator_settings(mf, orc, kw):
    inst, sc, _ = synth.cfg3(2)
    run_both(mf, orc, inst, sc.sla[:3], sc.omega[:3], seed=5, **kw)


def test_ga_small_space_and_wide_model(mf, orc):
    inst = synth.cfg0(2)
    sc = synth.ga_scenarios(2, 5, seed=2)
    run_both(mf, orc, inst, sc.sla, sc.omega, pop=32, gens=10, seed=9)
    inst2 = synth.make_instance([6, 5, 4], 16, 6, 64, 64, seed=3, vram_quantile=0.5)
    sc2 = synth.ga_scenarios(3, 4, seed=4)
    run_both(mf, orc, inst2, sc2.sla, sc2.omega, pop=96, gens=6, seed=1)


def test_ga_no_feasible_configuration(mf, orc):
    inst = synth.cfg1(0)
    inst.vram_cap = 1.0
    sc = synth.ga_scenarios(5, 3, seed=0)
    p = mf.Problem(inst)
    # both fitness kernels: a small population, and 3 x 4096 individuals
    for pop in (16, 4096):
        g = p.ga(sc.sla, sc.omega, pop=pop, gens=2, final_pop=True)
        assert np.all(g["best_idx"] == np.uint64(2 ** 64 - 1)) and np.all(np.isneginf(g["best_J"]))
        assert np.all(g["final_pop"].cpu().numpy().astype(np.uint64) == np.uint64(2 ** 64 - 1))
    # and a problem with feasible configurations right after, on the same device
    inst2 = synth.cfg1(0)
    run_both(mf, orc, inst2, sc.sla, sc.omega, pop=16, gens=2, seed=3)


def test_ga_rejects_bad_arguments(mf):
    inst, sc, _ = synth.cfg3(0)
    p = mf.Problem(inst)
    for kw in [dict(pop=7), dict(pop=2), dict(tourn_k=0), dict(tourn_k=9), dict(gens=-1)]:
        with pytest.raises(mf.MfError) as e:
            p.ga(sc.sla[:2], sc.omega[:2], **kw)
        assert e.value.status == mf.MF_EINVAL


def run_both_obj(mf, orc, inst, sla, omega, ob, st, **kw):
    print(f"[ga] {inst.name} S={len(sla)} eq3={ob is not None} fixed={st is not None} {kw}", flush=True)
    g = mf.Problem(inst, variants=ob).ga(sla, omega, final_pop=True, objective=ob, state=st, **kw)
    r = orc.Problem(inst, ob, state=st).ga(sla, omega, final_pop=True, **kw)
    np.testing.assert_array_equal(g["best_idx"], r["best_idx"])
    assert g["best_J"].tobytes() == r["best_J"].tobytes()
    np.testing.assert_array_equal(g["final_pop"].cpu().numpy().astype(np.uint64), r["final_pop"])
    return g, r


def test_ga_fixed_state_eq3(mf, orc):
    # the paper's GA setting (Section IV-C): population 100, 30 generations,
    # crossover 0.7, mutation 0.1, tournament 3, with the observed state
    # held fixed and the full utility of Eq. 3
    inst = synth.cfg1(0)
    ob = synth.make_objective(inst, 0)
    st = synth.make_state(inst, 0)
    sc = synth.ga_scenarios(5, 6, seed=1)
    g, r = run_both_obj(mf, orc, inst, sc.sla, sc.omega, ob, st, pop=100, gens=30, p_mut=0.1, seed=3)
    p = mf.Problem(inst, variants=ob)
    for s in range(6):
        ex = p.search(sc.sla[s], sc.omega[s], k=1, objective=ob, state=st)
        assert g["best_J"][s] <= ex["top_J"][0]


def test_ga_objective_and_state_apart(mf, orc):
    inst = synth.cfg1(2)
    sc = synth.ga_scenarios(5, 3, seed=2)
    run_both_obj(mf, orc, inst, sc.sla, sc.omega, synth.make_objective(inst, 2), None, pop=64, gens=8, seed=7)
    run_both_obj(mf, orc, inst, sc.sla, sc.omega, None, synth.make_state(inst, 2), pop=64, gens=8, seed=8)
    bf = synth.make_instance([7, 9, 3, 5], 8, 4, 64, 64, seed=9, vram_quantile=0.7, dtype="bf16")
    sc2 = synth.ga_scenarios(4, 2, seed=9)
    run_both_obj(mf, orc, bf, sc2.sla, sc2.omega, synth.make_objective(bf, 9), synth.make_state(bf, 9),
                 pop=32, gens=5, seed=2)


def test_ga_small_population_shapes(mf, orc):
    # small populations take the one-workgroup-per-individual fitness kernel:
    # more models than waves (two rounds, idle waves in the second), weights
    # staged in LDS and weights too large for it, a ragged last round
    sm = synth.make_instance([3, 2, 3, 2, 3, 2, 3, 2, 3, 2], 8, 4, 16, 16, seed=4, vram_quantile=0.8)
    sc = synth.ga_scenarios(10, 3, seed=4)
    run_both_obj(mf, orc, sm, sc.sla, sc.omega, synth.make_objective(sm, 4), synth.make_state(sm, 4),
                 pop=24, gens=6, seed=5)
    big = synth.make_instance([4, 3, 2, 3, 2, 3, 2, 3, 4], 16, 4, 128, 128, seed=5, vram_quantile=0.8)
    sc2 = synth.ga_scenarios(9, 2, seed=5)
    run_both_obj(mf, orc, big, sc2.sla, sc2.omega, synth.make_objective(big, 5), None, pop=16, gens=4, seed=6)
    run_both(mf, orc, big, sc2.sla, sc2.omega, pop=10, gens=3, seed=7)


def test_ga_largest_operator_footprint(mf, orc):
    # sixteen models, tournaments of eight, the largest population: the
    # operator kernel's largest LDS layout (population, every Philox word of
    # 64 pairs, parents' genes)
    inst = synth.make_instance([2] * 16, 8, 4, 16, 16, seed=6, vram_quantile=0.7)
    sc = synth.ga_scenarios(16, 1, seed=6)
    run_both(mf, orc, inst, sc.sla, sc.omega, pop=4096, gens=2, tourn_k=8, p_mut=0.2, seed=11)


def test_ga_large_population_shapes(mf, orc):
    # populations above 8,192 take the one-lane-per-individual fitness: the
    # paper's 64-32 sigmoid predictor with Eq. 3 and a fixed state, 22 inputs
    # at 64-64, 14 inputs at 32-32; ragged last workgroups
    a = synth.make_instance([12, 12, 9, 9, 9], 8, 4, 64, 32, seed=11, vram_quantile=0.8, act="sigmoid")
    sa = synth.ga_scenarios(5, 3, seed=11)
    run_both_obj(mf, orc, a, sa.sla, sa.omega, synth.make_objective(a, 11), synth.make_state(a, 11),
                 pop=2750, gens=3, p_mut=0.1, seed=12)
    b = synth.make_instance([6, 5, 4], 16, 6, 64, 64, seed=12, vram_quantile=0.7)
    sb = synth.ga_scenarios(3, 5, seed=12)
    run_both(mf, orc, b, sb.sla, sb.omega, pop=1700, gens=2, seed=13)
    c = synth.make_instance([7, 9, 3, 5], 10, 4, 32, 32, seed=13, vram_quantile=0.75)
    sc = synth.ga_scenarios(4, 3, seed=13)
    run_both_obj(mf, orc, c, sc.sla, sc.omega, synth.make_objective(c, 13), None, pop=3000, gens=3, seed=14)


def test_ga_memo_across_runs_and_forward_count(mf, orc):
    # large populations keep a memo of canonical predictions per joint index
    # for the run: later generations read it.  Runs on one problem reuse its
    # workspace (the memo starts empty every run); every run still equals the
    # oracle's replay, and the count of individuals that ran the surrogates
    # lies between one generation and all of them.
    inst, sc, gp = synth.cfg3(3)
    p = mf.Problem(inst)
    kw = dict(pop=2048, gens=30, tourn_k=3, p_cx=0.7, p_swap=0.5, p_mut=0.05)
    first = None
    for rows, seed in ((slice(0, 6), 1), (slice(6, 12), 2), (slice(0, 6), 1)):
        sla, om = sc.sla[rows], sc.omega[rows]
        print(f"[ga memo] rows={rows} seed={seed}", flush=True)
        g = p.ga(sla, om, final_pop=True, seed=seed, **kw)
        r = orc.Problem(inst).ga(sla, om, final_pop=True, seed=seed, **kw)
        np.testing.assert_array_equal(g["best_idx"], r["best_idx"])
        assert g["best_J"].tobytes() == r["best_J"].tobytes()
        np.testing.assert_array_equal(g["final_pop"].cpu().numpy().astype(np.uint64), r["final_pop"])
        n_gen = 6 * kw["pop"]
        assert n_gen <= g["forwards"] < n_gen * (kw["gens"] + 1) // 2, g["forwards"]
        if first is None:
            first = g
        elif seed == 1:
            assert g["forwards"] == first["forwards"]
            np.testing.assert_array_equal(g["best_idx"], first["best_idx"])
    # small populations evaluate every individual
    small = p.ga(sc.sla[:2], sc.omega[:2], pop=64, gens=4, seed=3)
    assert small["forwards"] == 2 * 64 * 5
