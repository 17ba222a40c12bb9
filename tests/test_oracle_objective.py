"""Pins for the oracle's full utility (Section II, Eq. 3) and throughput floor.

  * a hand-computed instance (the one of test_oracle.py) with dyadic
    parameters, values worked out below;
  * the special case that reduces Eq. 3 to the linear objective (Q = 1,
    extremes (0, 1), no reload, no penalty, no floor): bit-identical J;
  * the reload term alone: closed-form histogram of J over the whole space;
  * the floor alone: the feasible sets are nested in tau, with the linear
    feasible set at tau = -inf and none at a floor no output reaches;
  * the soft penalty alone: every feasible J lies in [-N beta delta^2, 0].
"""
from collections import Counter
from dataclasses import replace

import numpy as np

from paper_2609_02109_amd import synth
from test_oracle import HAND_THR, hand_instance


def hand_objective(tau=(0.0, 0.25)):
    # variant = option; model 0 was on variant 1, model 1 on variant 0
    V = synth.MAX_VARIANTS
    fmin = np.zeros((2, V), np.float32)
    fmax = np.ones((2, V), np.float32)
    qual = np.zeros((2, V), np.float32)
    fmin[0, :2] = (0, 1)
    fmax[0, :2] = (16, 17)
    fmax[1, :2] = (2, 4)
    qual[0, :2] = (1.0, 0.5)
    qual[1, :2] = (1.0, 0.75)
    return synth.Objective(variant=np.array([0, 1, 0, 1], np.int32), n_variants=np.array([2, 2], np.int32),
                           fmin=fmin, fmax=fmax, quality=qual, reload_cost=np.array([30, 5], np.float32),
                           prev_variant=np.array([1, 0], np.int32), tau=np.array(tau, np.float32),
                           alpha=1 / 64, beta=4.0, delta=0.125)


# Worked by hand (thr from test_oracle.py: idx 0 -> (1, 1), idx 1 -> (9, 2)):
# idx 0 = (0,0): model 0 variant 0: f = 1/16, q = 1/16, reload 30/64 (was on
#   variant 1), d = 1/8 - 1/16 > 0: penalty 4/256.  model 1 variant 0:
#   f = 1/2 >= 1/4, q = 1/2, no reload, d < 0.
#   J = 1/16 - 30/64 - 1/64 + 1/2 = 5/64 = 0.078125
# idx 1 = (0,1): model 0: f = 9/16, q = 9/16, reload 30/64, d < 0.  model 1
#   variant 1: f = 2/4 = 1/2, q = 3/4 * 1/2 = 3/8, reload 5/64, d < 0.
#   J = 9/16 - 30/64 + 3/8 - 5/64 = 25/64 = 0.390625
# idx 2 misses model 0's latency bound, idx 3 the VRAM cap.
def test_eq3_hand_values(orc):
    inst = hand_instance()
    r = orc.Problem(inst, hand_objective()).search(inst.sla, inst.omega, k=4, dump=True)
    np.testing.assert_array_equal(r["pred"][:, :, 1], HAND_THR)
    assert r["n_feas"] == 2
    assert list(r["top_idx"]) == [1, 0]
    assert list(r["top_J"]) == [25 / 64, 5 / 64]


def test_eq3_hand_floor_is_inclusive_and_penalised(orc):
    inst = hand_instance()
    # model 1 at f = 1/2 exactly on a floor of 1/2: feasible, and inside the
    # margin delta, so penalised by beta (1/2 + 1/8 - 1/2)^2 = 4/64
    r = orc.Problem(inst, hand_objective(tau=(0.0, 0.5))).search(inst.sla, inst.omega, k=4, dump=True)
    assert r["n_feas"] == 2
    assert list(r["top_J"]) == [25 / 64 - 4 / 64, 5 / 64 - 4 / 64]
    # a floor above 1/2 makes both configurations infeasible (model 1 misses it)
    r = orc.Problem(inst, hand_objective(tau=(0.0, 0.5001))).search(inst.sla, inst.omega, k=4, dump=True)
    assert r["n_feas"] == 0
    assert int(r["flags"][0]) & (1 << 9) and not int(r["flags"][0]) & (1 << 8)


def test_eq3_reduces_to_linear(orc):
    for inst in (synth.cfg1(0), synth.make_instance([5, 4, 3], 8, 8, 64, 64, seed=3, vram_quantile=0.6,
                                                    sla_range=(-0.3, 0.8), dtype="bf16")):
        a = orc.Problem(inst).search(inst.sla, inst.omega, k=16, dump=True)
        b = orc.Problem(inst, synth.linear_objective(inst)).search(inst.sla, inst.omega, k=16, dump=True)
        assert a["J"].tobytes() == b["J"].tobytes()
        np.testing.assert_array_equal(a["flags"], b["flags"])
        assert list(a["top_idx"]) == list(b["top_idx"])


def test_eq3_reload_term_closed_form(orc):
    # Q = 0, no penalty, no floor, alpha = 1, c_i = 2^i: J = -sum_i 2^i eta_i,
    # so each J value is one pattern of changed models; its count over the
    # whole space is the product, per model, of the options that keep /
    # change the previous variant
    inst = synth.make_instance([6, 4, 9], seed=2, vram_cap=1e9, sla_range=(1e9, 1e9))
    ob = synth.make_objective(inst, seed=5)
    ob = replace(ob, quality=np.zeros_like(ob.quality), reload_cost=np.array([1, 2, 4], np.float32),
                 tau=np.full(3, -np.inf, np.float32), alpha=1.0, beta=0.0)
    r = orc.Problem(inst, ob).search(inst.sla, inst.omega, k=1, dump=True)
    assert r["n_feas"] == inst.space_size
    got = Counter(r["J"].tolist())
    offs = np.concatenate([[0], np.cumsum(inst.n_options)])
    same = [int(np.sum(ob.variant[offs[i]:offs[i + 1]] == ob.prev_variant[i])) for i in range(3)]
    want = Counter()
    for mask in range(8):
        cnt = 1
        for i in range(3):
            changed = (mask >> i) & 1
            cnt *= (int(inst.n_options[i]) - same[i]) if changed else same[i]
        if cnt:
            want[-float(mask)] += cnt
    assert got == want
    # the best configuration keeps every variant: the lowest such index
    digits = np.array(np.unravel_index(np.arange(inst.space_size), tuple(int(k) for k in inst.n_options))).T
    keep = np.all(ob.variant[offs[:-1] + digits] == ob.prev_variant, axis=1)
    assert r["top_idx"][0] == np.flatnonzero(keep)[0] and r["top_J"][0] == 0.0


def test_eq3_floor_nesting(orc):
    inst = synth.cfg1(1)
    base = synth.make_objective(inst, seed=1)
    lin = orc.Problem(inst).search(inst.sla, inst.omega)["n_feas"]
    counts = []
    for t in (-np.inf, -0.5, 0.0, 0.2, 0.35, 0.5, 1e30):
        ob = replace(base, tau=np.full(inst.n_models, t, np.float32))
        counts.append(orc.Problem(inst, ob).search(inst.sla, inst.omega)["n_feas"])
    assert counts[0] == lin
    assert all(a >= b for a, b in zip(counts, counts[1:]))
    assert counts[-1] == 0 and counts[2] < counts[0]
    # nested sets, not only counts: every config feasible at 0.35 is feasible at 0.2
    f20 = orc.Problem(inst, replace(base, tau=np.full(5, 0.2, np.float32))).search(
        inst.sla, inst.omega, dump=True)["flags"]
    f35 = orc.Problem(inst, replace(base, tau=np.full(5, 0.35, np.float32))).search(
        inst.sla, inst.omega, dump=True)["flags"]
    assert not np.any((f35 & orc.FLAG_FEAS) & ~(f20 & orc.FLAG_FEAS))


def test_eq3_penalty_range(orc):
    inst = synth.cfg1(2)
    ob = replace(synth.make_objective(inst, seed=2), quality=np.zeros((5, synth.MAX_VARIANTS), np.float32),
                 alpha=0.0)
    r = orc.Problem(inst, ob).search(inst.sla, inst.omega, dump=True)
    J = r["J"][(r["flags"] & orc.FLAG_FEAS) != 0]
    assert len(J) > 0
    assert np.all(J <= 0.0) and np.all(J >= -inst.n_models * ob.beta * ob.delta ** 2 * (1 + 1e-12))
    assert np.any(J < 0.0) and np.any(J == 0.0)
    assert np.all(np.isneginf(r["J"][(r["flags"] & orc.FLAG_FEAS) == 0]))
