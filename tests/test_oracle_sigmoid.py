"""Pins for the sigmoid output of the surrogate (Section III-B: the
predictor's output layer is a sigmoid) in the oracle.

  * the oracle's e^x against libm's exp over [-700, 700]: within 2 units of
    2^-53 relative, exact at 0;
  * sigmoid(0) = 1/2 exactly, monotone on a dense grid, sigmoid(y) +
    sigmoid(-y) = 1 to rounding, clamped beyond +-700;
  * torch's float64 sigmoid (a library routine) agrees within 4 units of
    2^-53;
  * a sigmoid-output instance predicts exactly the oracle's sigmoid of the
    identity instance's outputs (the activation follows layer 3, on both
    outputs, and changes nothing else).
"""
import math
from dataclasses import replace

import numpy as np

from paper_2609_02109_amd import synth


def test_exp_against_libm(orc):
    xs = np.concatenate([np.linspace(-700, 700, 40_001), np.linspace(-1, 1, 10_001), [0.0, 1e-300, -1e-300]])
    worst = 0.0
    for x in xs:
        a, b = orc.exp(float(x)), math.exp(float(x))
        worst = max(worst, abs(a - b) / b)
    assert worst <= 2 * 2.0 ** -53
    assert orc.exp(0.0) == 1.0


def test_sigmoid_properties(orc):
    assert orc.sigmoid(0.0) == 0.5
    ys = np.linspace(-60, 60, 60_001)
    s = np.array([orc.sigmoid(float(y)) for y in ys])
    assert np.all(np.diff(s) >= 0.0)
    sm = np.array([orc.sigmoid(float(-y)) for y in ys])
    assert np.max(np.abs(s + sm - 1.0)) <= 2.0 ** -52
    assert orc.sigmoid(800.0) == orc.sigmoid(700.0) == 1.0
    assert orc.sigmoid(-800.0) == orc.sigmoid(-700.0) > 0.0


def test_sigmoid_against_torch(orc):
    import torch
    ys = np.linspace(-40, 40, 8_001)
    ref = torch.sigmoid(torch.from_numpy(ys)).numpy()
    got = np.array([orc.sigmoid(float(y)) for y in ys])
    assert np.max(np.abs(got - ref) / ref) <= 4 * 2.0 ** -53


def test_sigmoid_instance_applies_the_activation_after_layer3(orc):
    inst = synth.make_instance([5, 4, 6], 8, 4, 32, 32, seed=3, vram_cap=1e9, sla_range=(0.6, 0.95), act="sigmoid")
    ident = replace(inst, act="identity")
    idx = np.arange(inst.space_size, dtype=np.uint64)
    a = orc.Problem(inst).eval_list(idx, inst.sla, inst.omega)
    b = orc.Problem(ident).eval_list(idx, np.full(3, np.inf, np.float32), inst.omega)
    sig = np.vectorize(orc.sigmoid)
    assert a["lat"].tobytes() == sig(b["lat"]).tobytes()
    assert a["thr"].tobytes() == sig(b["thr"]).tobytes()
    assert np.all((a["lat"] > 0) & (a["lat"] < 1))
    # bounds at each model's median latency: the mask follows the sigmoid
    # outputs, inclusive
    sla = np.median(a["lat"], axis=0).astype(np.float32)
    m = orc.Problem(inst).eval_list(idx, sla, inst.omega)
    assert ((m["flags"] & orc.FLAG_SLA) != 0).tolist() == np.all(a["lat"] <= sla.astype(np.float64), axis=1).tolist()
    assert 0 < int(((m["flags"] & orc.FLAG_FEAS) != 0).sum()) < len(idx)
