"""GPU parity of the search with the observed state held fixed (Section
III-B: the aggregate state the surrogates see is observed and held fixed
during the search), against the CPU oracle's fixed-state mode, through the C
ABI.

Bars: VRAM / service / feasible masks, n_vram, n_feas, top-k indices and
canonical J bit-exact; the dumped predictions are the canonical values
rounded to fp32, so they equal the oracle's rounded to fp32 bit for bit.  At
the full sizes (the whole joint space) the exact counts come from an
independent meet-in-the-middle count over the oracle's per-option values,
and the top-k from the oracle's evaluation of the returned indices.
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


def fixed_parity(mf, orc, inst, state, lo, hi, k, ob=None):
    print(f"[fixed] {inst.name} seed={inst.seed} range=[{lo},{hi}) k={k} eq3={ob is not None}", flush=True)
    p = mf.Problem(inst, variants=ob)
    g = p.search(inst.sla, inst.omega, k=k, lo=lo, hi=hi, dump=True, objective=ob, state=state)
    r = orc.Problem(inst, ob, state=state).search(inst.sla, inst.omega, k=k, lo=lo, hi=hi, dump=True)
    assert g["n_eval"] == hi - lo
    assert g["n_vram"] == r["n_vram"]
    assert g["n_feas"] == r["n_feas"]
    assert g["n_flagged"] == 0 and g["n_topk_collect"] == 0 and g["n_splits"] == 0
    gm = g["mask"].cpu().numpy().astype(np.uint32)
    rf = r["flags"]
    np.testing.assert_array_equal(gm & 7, rf & 7)
    assert not np.any(gm & 8)
    np.testing.assert_array_equal(g["top_idx"], r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()
    assert g["pred"].cpu().numpy().tobytes() == r["pred"].astype(np.float32).tobytes()
    p.close()
    return g, r


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_fixed_n5_full(mf, orc, seed):
    inst = synth.cfg1(seed)
    g, r = fixed_parity(mf, orc, inst, synth.make_state(inst, seed), 0, inst.space_size, 16)
    assert 0 < r["n_feas"] <= r["n_vram"]


def test_fixed_n2_full(mf, orc):
    inst = synth.cfg0(2)
    fixed_parity(mf, orc, inst, synth.make_state(inst, 2), 0, inst.space_size, 1)


@pytest.mark.parametrize("seed", [0, 1])
def test_fixed_eq3_n5_full(mf, orc, seed):
    inst = synth.cfg1(seed)
    g, r = fixed_parity(mf, orc, inst, synth.make_state(inst, seed), 0, inst.space_size, 16,
                        synth.make_objective(inst, seed))
    assert r["n_feas"] > 0


# Shapes whose last two models form the scanned inner block with a periodic
# last digit (its option count 3 x 2^j, 128 or 2^j): whole-space searches
# without a dump take the scan that keeps each lane's rows of the last model
# in registers.  Counts, top-k indices and canonical J against the oracle.
# (instance seeds with feasible configurations under both objectives)
@pytest.mark.parametrize("n_options,period,seed", [([5, 16, 24], 3, 0), ([3, 2, 128], 2, 3), ([7, 16, 16], 1, 0),
                                                   ([2, 4, 8, 48], 3, 0), ([5, 24, 24], 3, 0), ([3, 16, 32], 1, 0)])
@pytest.mark.parametrize("eq3", [False, True])
def test_fixed_periodic_last_digit(mf, orc, n_options, period, seed, eq3):
    inst = synth.make_instance(n_options, 8, 4, 32, 32, seed=seed, vram_quantile=0.7)
    state = synth.make_state(inst, 3)
    ob = synth.make_objective(inst, 3) if eq3 else None
    k = 8 if eq3 else 16
    print(f"[fixed periodic] K={n_options} eq3={eq3}", flush=True)
    p = mf.Problem(inst, variants=ob)
    g = p.search(inst.sla, inst.omega, k=k, objective=ob, state=state)
    r = orc.Problem(inst, ob, state=state).search(inst.sla, inst.omega, k=k, lo=0, hi=inst.space_size)
    p.close()
    assert g["n_vram"] == r["n_vram"] and g["n_feas"] == r["n_feas"]
    assert 0 < r["n_feas"] < inst.space_size
    np.testing.assert_array_equal(g["top_idx"], r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()


# Whole spaces of 6-9 million configurations with a periodic last digit:
# several blocks per wave, so a wave's list fills and the later blocks whose
# largest possible J falls under its k-th J form only the counts.  Any block
# skipped wrongly would drop a configuration of the oracle's exact top-k.
@pytest.mark.parametrize("n_options", [[24, 32, 32, 16, 16], [16, 32, 32, 24, 24]])
@pytest.mark.parametrize("eq3", [False, True])
def test_fixed_periodic_pruned_blocks(mf, orc, n_options, eq3):
    inst = synth.make_instance(n_options, 8, 4, 32, 32, seed=0, vram_quantile=0.7)
    state = synth.make_state(inst, 3)
    ob = synth.make_objective(inst, 3) if eq3 else None
    k = 8
    print(f"[fixed pruned] K={n_options} eq3={eq3}", flush=True)
    p = mf.Problem(inst, variants=ob)
    g = p.search(inst.sla, inst.omega, k=k, objective=ob, state=state)
    p.close()
    r = orc.Problem(inst, ob, state=state).search(inst.sla, inst.omega, k=k, lo=0, hi=inst.space_size)
    assert g["n_vram"] == r["n_vram"] and g["n_feas"] == r["n_feas"]
    assert r["n_feas"] > 100_000
    np.testing.assert_array_equal(g["top_idx"], r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_fixed_n6_ranges(mf, orc):
    inst = synth.cfg2(0)
    st = synth.make_state(inst, 0)
    n = inst.space_size
    fixed_parity(mf, orc, inst, st, 0, 100_000, 8)
    fixed_parity(mf, orc, inst, st, n // 2 - 33_333, n // 2 + 30_001, 8, synth.make_objective(inst, 0))
    fixed_parity(mf, orc, inst, st, n - 40_001, n, 4)


def test_fixed_bf16(mf, orc):
    inst = synth.make_instance([7, 9, 3, 5], 12, 8, 128, 128, seed=9, vram_quantile=0.7, sla_range=(0.0, 1.0),
                               dtype="bf16")
    fixed_parity(mf, orc, inst, synth.make_state(inst, 9), 0, inst.space_size, 9)
    inst8 = synth.cfg4(1)
    fixed_parity(mf, orc, inst8, synth.make_state(inst8, 1), 2 ** 31 - 5_000, 2 ** 31 + 5_000, 64,
                 synth.make_objective(inst8, 1))


def test_fixed_shape_without_fast_kernel(mf, orc):
    # H1 != H2 and an fp32 width with no fast kernel: the derived-state search
    # rejects the shape, the fixed-state search runs it
    inst = synth.make_instance([5, 7, 4, 6], 8, 6, 48, 40, seed=5, vram_quantile=0.7, sla_range=(-0.2, 0.9))
    p = mf.Problem(inst)
    with pytest.raises(mf.MfError) as e:
        p.search(inst.sla, inst.omega, k=4)
    assert e.value.status == mf.MF_EUNSUPPORTED
    fixed_parity(mf, orc, inst, synth.make_state(inst, 5), 0, inst.space_size, 12)


def test_fixed_degenerate_ranges_and_validation(mf, orc):
    inst = synth.cfg1(1)
    st = synth.make_state(inst, 1)
    p = mf.Problem(inst)
    g = p.search(inst.sla, inst.omega, k=5, lo=77, hi=77, state=st)
    assert g["n_eval"] == 0 and g["n_feas"] == 0 and len(g["top_idx"]) == 0
    for lo in (0, 4321, inst.space_size - 1):
        fixed_parity(mf, orc, inst, st, lo, lo + 1, 3)
    # k larger than the feasible set: every feasible configuration, sorted
    tight = replace(inst, sla=np.full(inst.n_models, -1e9, np.float32))
    g = mf.Problem(tight).search(tight.sla, tight.omega, k=64, state=st)
    assert g["n_feas"] == 0 and len(g["top_idx"]) == 0
    bad = st.copy()
    bad[1] = np.nan
    with pytest.raises(mf.MfError) as e:
        p.search(inst.sla, inst.omega, k=1, state=bad)
    assert e.value.status == mf.MF_EINVAL
    with pytest.raises(ValueError):
        p.search(inst.sla, inst.omega, k=1, state=st[:-1])


def test_fixed_topk_ties(mf, orc):
    # throughput independent of the option: every feasible configuration
    # ties at J = sum omega, far more than k; the lowest indices win
    inst = synth.make_instance([12, 11, 10], 8, 4, 64, 64, seed=4, vram_quantile=0.7, sla_range=(0.2, 1.0))
    for i in range(inst.n_models):
        W1, b1, W2, b2, W3, b3 = inst.model_weights(i)
        W3[1, :] = 0.0
        b3[1] = 1.0
    g, r = fixed_parity(mf, orc, inst, synth.make_state(inst, 4), 0, inst.space_size, 64)
    assert r["n_feas"] > 64


def row_values(orc, inst, state, ob=None):
    """Per option row of each model: (row ok, thr) from the oracle, evaluated
    on one configuration per row (model i at option o, the others at 0)."""
    K = [int(x) for x in inst.n_options]
    N = len(K)
    idx = []
    for i in range(N):
        for o in range(K[i]):
            d = [0] * N
            d[i] = o
            idx.append(int(np.ravel_multi_index(tuple(d), tuple(K))))
    r = orc.Problem(inst, ob, state=state).eval_list(np.array(idx, np.uint64), inst.sla, inst.omega)
    ok, thr, t = [], [], 0
    for i in range(N):
        ok.append(np.array([not (int(r["flags"][t + o]) >> (8 + i)) & 1 for o in range(K[i])]))
        thr.append(r["thr"][t:t + K[i], i].copy())
        t += K[i]
    return ok, thr


def meet_in_the_middle(inst, ok, thr):
    """Exact feasible and VRAM-feasible counts, and the best J up to fp64
    rounding, of the linear objective over the whole space (sorted half-space
    VRAM sums; the sums are exact on the 2^-14 grid)."""
    K = [int(x) for x in inst.n_options]
    N = len(K)
    offs = np.concatenate([[0], np.cumsum(K)])
    vram = [inst.features[offs[i]:offs[i + 1], inst.agg_cols[inst.vram_slot]].astype(np.float64) for i in range(N)]

    def half(models):
        v, j, a = np.zeros(1), np.zeros(1), np.zeros(1)
        good = np.ones(1, bool)
        for i in models:
            w = float(inst.omega[i]) * thr[i]
            v = (v[:, None] + vram[i][None, :]).ravel()
            j = (j[:, None] + w[None, :]).ravel()
            a = (a[:, None] + np.abs(w)[None, :]).ravel()
            good = (good[:, None] & ok[i][None, :]).ravel()
        return v, j, a, good

    v1, j1, a1, g1 = half(range(N // 2))
    v2, j2, a2, g2 = half(range(N // 2, N))
    cap = float(inst.vram_cap)
    v2s = np.sort(v2)
    n_vram = int(np.searchsorted(v2s, cap - v1, side="right").sum())
    v1g, j1g, a1g = v1[g1], j1[g1], a1[g1]
    o = np.argsort(v2[g2], kind="stable")
    v2g, j2g, a2g = v2[g2][o], j2[g2][o], a2[g2][o]
    cut = np.searchsorted(v2g, cap - v1g, side="right")
    n_feas = int(cut.sum())
    pref = np.maximum.accumulate(j2g)
    arg = np.zeros(len(pref), np.int64)
    for t in range(1, len(pref)):
        arg[t] = t if j2g[t] > pref[t - 1] else arg[t - 1]
    has = cut > 0
    cand = np.where(has, j1g + pref[np.maximum(cut - 1, 0)], -np.inf)
    q = int(np.argmax(cand))
    best = float(cand[q])
    scale = float(a1g[q] + a2g[arg[cut[q] - 1]]) if has.any() else 0.0
    return n_vram, n_feas, best, scale


@pytest.mark.parametrize("which", ["n6", "n8"])
def test_fixed_full_space_properties(mf, orc, which):
    inst = synth.cfg2(0) if which == "n6" else synth.cfg4(0)
    st = synth.make_state(inst, 3)
    k = 64
    print(f"[fixed] full space {inst.name} {inst.space_size}", flush=True)
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=k, state=st)
    assert g["n_eval"] == inst.space_size
    ok, thr = row_values(orc, inst, st)
    n_vram, n_feas, best, scale = meet_in_the_middle(inst, ok, thr)
    assert g["n_vram"] == n_vram
    assert g["n_feas"] == n_feas
    assert len(g["top_idx"]) == min(k, n_feas) > 0
    top = np.asarray(g["top_idx"], np.uint64)
    ref = orc.Problem(inst, state=st).eval_list(top, inst.sla, inst.omega)
    assert np.all(ref["flags"] & 4)
    assert g["top_J"].tobytes() == ref["J"].tobytes()
    keys = list(zip(-g["top_J"], top.tolist()))
    assert keys == sorted(keys)
    assert abs(g["top_J"][0] - best) <= 4 * inst.n_models * 2.0 ** -52 * scale
    # no sampled feasible configuration beats the k-th
    rng = np.random.default_rng(11)
    samp = rng.integers(0, inst.space_size, 3_000, dtype=np.int64).astype(np.uint64)
    rs = orc.Problem(inst, state=st).eval_list(samp, inst.sla, inst.omega)
    feas = (rs["flags"] & 4) != 0
    kth = g["top_J"][-1]
    in_top = np.isin(samp, top)
    assert np.all((rs["J"][feas] < kth) | ((rs["J"][feas] == kth) & (samp[feas] >= top[-1])) | in_top[feas])


def test_fixed_eq3_full_space_counts(mf, orc):
    # the floors and latency bounds per row decide feasibility: the counts
    # over the whole N=8 space follow from the per-row decisions exactly
    inst = synth.cfg4(2)
    st = synth.make_state(inst, 2)
    ob = synth.make_objective(inst, 2)
    g = mf.Problem(inst, variants=ob).search(inst.sla, inst.omega, k=64, objective=ob, state=st)
    ok, thr = row_values(orc, inst, st, ob)
    n_vram, n_feas, _, _ = meet_in_the_middle(inst, ok, thr)
    assert g["n_vram"] == n_vram and g["n_feas"] == n_feas > 0
    top = np.asarray(g["top_idx"], np.uint64)
    ref = orc.Problem(inst, ob, state=st).eval_list(top, inst.sla, inst.omega)
    assert np.all(ref["flags"] & 4)
    assert g["top_J"].tobytes() == ref["J"].tobytes()
    keys = list(zip(-g["top_J"], top.tolist()))
    assert keys == sorted(keys)
