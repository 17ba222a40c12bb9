"""Pins for the oracle's fixed-observed-state mode (Section III-B: the
aggregate state fed to the surrogates is observed and held fixed during the
search, so each model's prediction depends on its own option only).

  * invariance: model i's predictions do not move when other models change
    their option;
  * consistency: with the state set to a candidate's own aggregate, that
    candidate's predictions equal the derived-state ones bit for bit;
  * an independent meet-in-the-middle search (sorted half-space VRAM sums,
    prefix maxima) reproduces the feasible count exactly and the optimum J
    to fp64 rounding; the VRAM-feasible count is the derived mode's.
"""
import numpy as np

from paper_2609_02109_amd import synth


def test_fixed_state_predictions_depend_on_own_option(orc):
    inst = synth.cfg1(0)
    p = orc.Problem(inst, state=synth.make_state(inst, 0))
    r = p.search(inst.sla, inst.omega, dump=True)
    K = [int(k) for k in inst.n_options]
    digits = np.array(np.unravel_index(np.arange(inst.space_size), tuple(K))).T
    for i in range(inst.n_models):
        for o in range(K[i]):
            sel = r["pred"][digits[:, i] == o, i, :]
            assert np.all(sel == sel[0])
    # ... while with the derived aggregate they do move
    rd = orc.Problem(inst).search(inst.sla, inst.omega, dump=True)
    assert not np.all(rd["pred"][digits[:, 0] == 0, 0, 1] == rd["pred"][0, 0, 1])


def test_fixed_state_equals_derived_at_the_state_candidate(orc):
    inst = synth.make_instance([5, 4, 6], 8, 6, 64, 64, seed=4, vram_quantile=0.7, sla_range=(-0.3, 0.9))
    pd = orc.Problem(inst)
    for idx in (0, 37, inst.space_size - 1):
        a, exact = pd.aggregate(pd.decode(idx))
        assert exact
        lat_d, thr_d, J_d, f_d = pd.eval(idx, inst.sla, inst.omega)
        lat_f, thr_f, J_f, f_f = orc.Problem(inst, state=a).eval(idx, inst.sla, inst.omega)
        assert lat_d.tobytes() == lat_f.tobytes() and thr_d.tobytes() == thr_f.tobytes()
        assert J_d == J_f or (np.isinf(J_d) and np.isinf(J_f))


def test_fixed_state_meet_in_the_middle(orc):
    inst = synth.cfg1(2)
    st = synth.make_state(inst, 2)
    p = orc.Problem(inst, state=st)
    r = p.search(inst.sla, inst.omega, k=4, dump=True)
    K = [int(k) for k in inst.n_options]
    N = len(K)
    offs = np.concatenate([[0], np.cumsum(K)])
    # per-option predictions read from the dump, and each option's VRAM
    digits = np.array(np.unravel_index(np.arange(inst.space_size), tuple(K))).T
    thr = [np.zeros(k) for k in K]
    ok = [np.zeros(k, bool) for k in K]
    for i in range(N):
        for o in range(K[i]):
            t = int(np.flatnonzero(digits[:, i] == o)[0])
            thr[i][o] = r["pred"][t, i, 1]
            ok[i][o] = r["pred"][t, i, 0] <= float(inst.sla[i])
    vram = [inst.features[offs[i]:offs[i + 1], inst.agg_cols[inst.vram_slot]].astype(np.float64) for i in range(N)]

    def half(models):
        v = np.zeros(1)
        j = np.zeros(1)
        good = np.ones(1, bool)
        for i in models:
            v = (v[:, None] + vram[i][None, :]).ravel()
            j = (j[:, None] + float(inst.omega[i]) * thr[i][None, :]).ravel()
            good = (good[:, None] & ok[i][None, :]).ravel()
        return v[good], j[good]

    v1, j1 = half(range(N // 2))
    v2, j2 = half(range(N // 2, N))
    order = np.argsort(v2, kind="stable")
    v2s, j2s = v2[order], j2[order]
    pref = np.maximum.accumulate(j2s)
    cap = float(inst.vram_cap)
    cut = np.searchsorted(v2s, cap - v1, side="right")
    assert int(cut.sum()) == r["n_feas"]
    best = max(j1[q] + pref[c - 1] for q, c in enumerate(cut) if c > 0)
    assert abs(best - r["top_J"][0]) <= 1e-12 * abs(best)
    assert r["n_vram"] == orc.Problem(inst).search(inst.sla, inst.omega)["n_vram"]
