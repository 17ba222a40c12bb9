"""Pins for the GA oracle (oracle/mf_oracle_ga.c), against facts fixed outside it.

  * Philox4x64-10 against numpy.random.Philox (a library implementation);
  * outcome: the GA's best is feasible, its J is reproduced by the canonical
    evaluation, and it never beats the exhaustive optimum (the exhaustive
    search is the upper bound of every scheduler on the same landscape,
    Section IV-C); on a 36-configuration space it finds the optimum;
  * operator laws, measured statistically on ga_next:
      elitism keeps the best individual in slot 0;
      a tournament of k draws with replacement selects the individual of rank
        r (0 = best of P) with probability ((P-r)/P)^k - ((P-r-1)/P)^k;
      mutation changes a gene with probability p_mut (K-1)/K, uniformly;
      uniform crossover mixes parents only gene-wise;
      repair leaves every individual VRAM-feasible;
      the initial population is uniform over the feasible list.
"""
import numpy as np
import pytest
from scipy import stats

from paper_2609_02109_amd import synth


def np_philox(ctr, key):
    mask = (1 << 64) - 1
    c = sum(int(v) << (64 * i) for i, v in enumerate(ctr))
    c = (c - 1) % (1 << 256)   # numpy increments the counter before each block
    cc = np.array([(c >> (64 * i)) & mask for i in range(4)], dtype=np.uint64)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=cc)
    return [int(v) for v in bg.random_raw(4)]


def test_philox_matches_numpy(orc):
    rng = np.random.default_rng(0)
    for _ in range(300):
        ctr = [int(v) for v in rng.integers(0, 2 ** 63, 4, dtype=np.int64)]
        key = [int(v) for v in rng.integers(0, 2 ** 63, 2, dtype=np.int64)]
        assert orc.philox4x64(ctr, key) == np_philox(ctr, key)
    assert orc.philox4x64([0, 0, 0, 0], [0, 0]) == np_philox([0, 0, 0, 0], [0, 0])


def test_ga_outcome_bounded_by_exhaustive(orc):
    inst, sc, _ = synth.cfg3(0)
    p = orc.Problem(inst)
    S = 6
    r = p.ga(sc.sla[:S], sc.omega[:S], pop=256, gens=20, seed=3)
    for s in range(S):
        ex = p.search(sc.sla[s], sc.omega[s], k=1)
        assert r["best_J"][s] <= ex["top_J"][0]
        lat, thr, J, fl = p.eval(int(r["best_idx"][s]), sc.sla[s], sc.omega[s])
        assert fl & orc.FLAG_FEAS and J == r["best_J"][s]


def test_ga_finds_optimum_on_small_space(orc):
    inst = synth.cfg0(1)
    p = orc.Problem(inst)
    sc = synth.ga_scenarios(2, 4, seed=1)
    r = p.ga(sc.sla, sc.omega, pop=64, gens=15, seed=1)
    for s in range(4):
        ex = p.search(sc.sla[s], sc.omega[s], k=1)
        if len(ex["top_idx"]):
            assert int(r["best_idx"][s]) == int(ex["top_idx"][0])
            assert r["best_J"][s] == ex["top_J"][0]


def test_ga_deterministic_and_thread_independent(orc):
    inst, sc, _ = synth.cfg3(1)
    p = orc.Problem(inst)
    a = p.ga(sc.sla[:4], sc.omega[:4], pop=128, gens=10, seed=7, threads=1, final_pop=True)
    b = p.ga(sc.sla[:4], sc.omega[:4], pop=128, gens=10, seed=7, threads=8, final_pop=True)
    c = p.ga(sc.sla[:4], sc.omega[:4], pop=128, gens=10, seed=8, final_pop=True)
    assert np.array_equal(a["final_pop"], b["final_pop"]) and np.array_equal(a["best_J"], b["best_J"])
    assert not np.array_equal(a["final_pop"], c["final_pop"])
    # repair: every individual of the last population is VRAM-feasible
    fl = set(int(x) for x in p.vram_feasible())
    assert all(int(x) in fl for x in a["final_pop"].ravel())


def test_initial_population_uniform_over_feasible_list(orc):
    inst, sc, _ = synth.cfg3(0)
    p = orc.Problem(inst)
    fl = p.vram_feasible()
    r = p.ga(sc.sla, sc.omega, pop=2048, gens=0, seed=5, final_pop=True)
    pos = np.searchsorted(fl, r["final_pop"].ravel().astype(np.int64))
    assert np.all(fl[pos] == r["final_pop"].ravel())
    counts = np.bincount(pos * 64 // len(fl), minlength=64)
    assert stats.chisquare(counts).pvalue > 1e-4


def _distinct_population(p, inst, P, seed):
    fl = p.vram_feasible()
    rng = np.random.default_rng(seed)
    return fl, rng.choice(fl, P, replace=False).astype(np.uint64)


def test_elitism_and_tournament_law(orc):
    inst = synth.cfg1(0)
    p = orc.Problem(inst)
    P, k = 512, 3
    fl, pop = _distinct_population(p, inst, P, 0)
    rank = np.random.default_rng(1).permutation(P)          # rank 0 = best
    fit = (P - rank).astype(np.float64)
    slot_of = {int(x): j for j, x in enumerate(pop)}
    counts = np.zeros(P)
    for g in range(40):
        out = p.ga_next(0, g, pop, fit, fl, P, tourn_k=k, p_cx=0.0, p_mut=0.0, seed=11)
        assert int(out[0]) == int(pop[np.argmin(rank)])     # elitism
        for x in out[1:]:
            counts[rank[slot_of[int(x)]]] += 1               # children copy winners
    r = np.arange(P)
    prob = ((P - r) / P) ** k - ((P - r - 1) / P) ** k
    buckets = np.array_split(np.arange(P), 16)
    obs = np.array([counts[b].sum() for b in buckets])
    exp = np.array([prob[b].sum() for b in buckets]) * counts.sum()
    assert stats.chisquare(obs, exp).pvalue > 1e-4
    assert obs[0] > obs[-1] * 20                              # best ranks dominate


def test_mutation_law(orc):
    inst = synth.make_instance([12, 12, 9, 9, 9], seed=2, vram_cap=1e9)
    p = orc.Problem(inst)
    P, pm = 1024, 0.3
    fl = p.vram_feasible()
    c0 = p.encode([3, 5, 1, 7, 2])
    pop = np.full(P, c0, np.uint64)
    fit = np.zeros(P)
    changed = np.zeros(5)
    values = [np.zeros(int(k)) for k in inst.n_options]
    n = 0
    for g in range(20):
        out = p.ga_next(0, g, pop, fit, fl, P, tourn_k=2, p_cx=0.7, p_mut=pm, seed=4)
        for x in out[1:]:
            d = p.decode(int(x))
            changed += d != np.array([3, 5, 1, 7, 2])
            for i, v in enumerate(d):
                values[i][v] += 1
            n += 1
    K = inst.n_options.astype(float)
    expect = pm * (K - 1) / K
    z = (changed / n - expect) / np.sqrt(expect * (1 - expect) / n)
    assert np.all(np.abs(z) < 5)
    for i, k in enumerate(inst.n_options):
        base = [3, 5, 1, 7, 2][i]
        others = np.delete(values[i], base)
        assert stats.chisquare(others).pvalue > 1e-4           # new value uniform


def test_crossover_mixes_genewise(orc):
    inst = synth.make_instance([12, 12, 9, 9, 9], seed=2, vram_cap=1e9)
    p = orc.Problem(inst)
    P = 1024
    fl = p.vram_feasible()
    A, B = [1, 2, 3, 4, 5], [7, 8, 6, 0, 1]
    ia, ib = p.encode(A), p.encode(B)
    pop = np.array([ia if j % 2 == 0 else ib for j in range(P)], np.uint64)
    fit = np.zeros(P)
    for pcx, expect_mixed in [(0.0, 0.0), (1.0, 0.5 * (1 - 2.0 ** (1 - 5)))]:
        mixed = n = 0
        for g in range(10):
            out = p.ga_next(0, g, pop, fit, fl, P, tourn_k=1, p_cx=pcx, p_swap=0.5, p_mut=0.0, seed=9)
            for x in out[1:]:
                d = list(p.decode(int(x)))
                assert all(d[i] in (A[i], B[i]) for i in range(5))
                mixed += d not in (A, B)
                n += 1
        assert abs(mixed / n - expect_mixed) < 5 * np.sqrt(0.25 / n) + 1e-12


def test_repair_keeps_population_feasible(orc):
    inst = synth.cfg1(2)
    p = orc.Problem(inst)
    P = 1024
    fl = p.vram_feasible()
    fls = set(int(x) for x in fl)
    _, pop = _distinct_population(p, inst, P, 3)
    fit = np.zeros(P)
    out = p.ga_next(0, 0, pop, fit, fl, P, tourn_k=3, p_cx=1.0, p_mut=1.0, seed=5)
    assert all(int(x) in fls for x in out)
