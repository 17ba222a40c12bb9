"""GPU parity of the bf16 search path (bf16 weights, fp32 accumulation)
against the CPU oracle, through the C ABI.

The first hidden layer is the canonical fp32 chain on both sides, so its
bfloat16 values agree exactly; the fast path differs from the canonical values
only by the fp32 accumulation of layers 2 and 3, which per-configuration
bounds cover.  Bars:
  * VRAM / latency / feasible masks, n_vram, n_feas, top-k indices and
    canonical J: bit-exact.
  * fast predictions: within 2e-2 relative (the bf16 tolerance), and in fact
    within 1e-4 relative to max(|oracle|, rms) by the path's design.
"""
import hashlib
import json
import os

import numpy as np
import pytest

from paper_2609_02109_amd import synth
from test_gpu_search import GOLDEN, check_predictions, run_range_parity
from test_oracle import mitm_vram_count

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2
TOL_DESIGN = 1e-4


@pytest.fixture(scope="module")
def mf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_02109_amd import mf as mfmod
    return mfmod


def bf16_parity(mf, orc, inst, lo, hi, k):
    g, r = run_range_parity(mf, orc, inst, lo, hi, k, tol=TOL_BF16)
    check_predictions(g["pred"].cpu().numpy(), r["pred"], tol=TOL_DESIGN)
    return g, r


@pytest.mark.parametrize("shape", [
    dict(n_options=[6, 5, 4], n_local=8, n_agg=4, hidden=64),
    dict(n_options=[7, 9, 3, 5], n_local=12, n_agg=8, hidden=128),
    dict(n_options=[11], n_local=8, n_agg=2, hidden=64),               # N = 1
    dict(n_options=[1, 13, 1, 6], n_local=8, n_agg=6, hidden=64),      # options count 1
    dict(n_options=[2] * 16, n_local=8, n_agg=4, hidden=64),           # N = 16
    dict(n_options=[5, 4, 3], n_local=32, n_agg=8, hidden=256),        # the N=8 workload's model shape
    dict(n_options=[3, 1, 2, 2, 1, 3, 2, 2], n_local=8, n_agg=4, hidden=64),   # N = 8 with one-option models
    dict(n_options=[2, 3, 2, 2, 3, 2, 2, 2], n_local=16, n_agg=6, hidden=128),  # N = 8, every count > 1
])
def test_bf16_full_space(mf, orc, shape):
    inst = synth.make_instance(shape["n_options"], shape["n_local"], shape["n_agg"], shape["hidden"],
                               shape["hidden"], seed=7, vram_quantile=0.6, sla_range=(-0.2, 0.8),
                               dtype="bf16")
    bf16_parity(mf, orc, inst, 0, inst.space_size, 9)


def test_bf16_n8_ragged_ranges(mf, orc):
    # the full N=8 shape (16 options per model, 40->256->256->2), top-64:
    # a head range, a range across the 2^31 midpoint and the ragged tail
    inst = synth.cfg4(0)
    n = inst.space_size
    bf16_parity(mf, orc, inst, 0, 20_000, 64)
    bf16_parity(mf, orc, inst, (n // 2) - 7_777, (n // 2) + 9_001, 64)
    bf16_parity(mf, orc, inst, n - 12_345, n, 64)


def test_bf16_layer1_values_exact(mf, orc):
    # W2 = I, b2 = 0, W3 picks one hidden unit per output: then lat = h1[u0]
    # and thr = h1[u1] exactly on both sides, so the fast predictions must
    # equal the oracle's bit for bit (an error in the fp32 chain order or in
    # the bfloat16 rounding of any tested unit shows up directly)
    inst = synth.make_instance([9, 8, 7], 8, 8, 64, 64, seed=12, vram_cap=1e9, sla_range=(50.0, 60.0),
                               dtype="bf16")
    units = [(0, 37), (5, 63), (31, 32)]
    for i in range(inst.n_models):
        W1, b1, W2, b2, W3, b3 = inst.model_weights(i)
        W2[:] = np.eye(64, dtype=np.float32)
        b2[:] = 0.0
        W3[:] = 0.0
        W3[0, units[i][0]] = 1.0
        W3[1, units[i][1]] = 1.0
        b3[:] = 0.0
    idx = np.arange(inst.space_size, dtype=np.int64)
    p = mf.Problem(inst)
    fast = p.eval_fast(idx).cpu().numpy().astype(np.float64)
    ref = orc.Problem(inst).eval_list(idx.astype(np.uint64), inst.sla, inst.omega)
    rp = np.stack([ref["lat"], ref["thr"]], axis=-1)
    assert np.count_nonzero(rp) > rp.size // 4
    np.testing.assert_array_equal(fast, rp)


def test_bf16_eval_sampled_full_size(mf, orc):
    inst = synth.cfg4(1)
    rng = np.random.default_rng(1)
    idx = rng.integers(0, inst.space_size, 3_000, dtype=np.int64)
    idx[:3] = [0, inst.space_size - 1, inst.space_size // 2]
    p = mf.Problem(inst)
    fast = p.eval_fast(idx).cpu().numpy()
    can = p.eval_canonical(idx, inst.sla, inst.omega)
    ref = orc.Problem(inst).eval_list(idx.astype(np.uint64), inst.sla, inst.omega)
    rp = np.stack([ref["lat"], ref["thr"]], axis=-1)
    check_predictions(fast, rp, tol=TOL_BF16)
    check_predictions(fast, rp, tol=TOL_DESIGN)
    assert can["pred"].cpu().numpy().tobytes() == rp.tobytes()
    assert can["J"].cpu().numpy().tobytes() == ref["J"].tobytes()


def test_bf16_n8_full_space_properties(mf, orc):
    # the whole 2^32-configuration space: the top-64 are feasible with the
    # oracle's J bit for bit, sorted by (J desc, index asc), and no sampled
    # feasible configuration, and no feasible configuration one option from a
    # top-64 member or two options from one of the best four, beats the 64th
    inst = synth.cfg4(0)
    print(f"[bf16] full N=8 space {inst.space_size}", flush=True)
    p = mf.Problem(inst)
    g = p.search(inst.sla, inst.omega, k=64)
    assert g["n_eval"] == inst.space_size
    assert len(g["top_idx"]) == 64 and 64 <= g["n_feas"] <= g["n_vram"]
    # the VRAM-feasible count over all 2^32 configurations, exactly (an
    # independent meet-in-the-middle count over the option tables)
    assert g["n_vram"] == mitm_vram_count(inst, float(inst.vram_cap))
    top = np.asarray(g["top_idx"], dtype=np.uint64)
    ref = orc.Problem(inst).eval_list(top, inst.sla, inst.omega)
    assert np.all(ref["flags"] & 4)
    assert g["top_J"].tobytes() == ref["J"].tobytes()
    keys = list(zip(-g["top_J"], top.tolist()))
    assert keys == sorted(keys)
    rng = np.random.default_rng(5)
    samp = rng.integers(0, inst.space_size, 4_000, dtype=np.int64).astype(np.uint64)
    rs = orc.Problem(inst).eval_list(samp, inst.sla, inst.omega)
    feas = (rs["flags"] & 4) != 0
    kth = g["top_J"][-1]
    in_top = np.isin(samp, top)
    assert np.all((rs["J"][feas] < kth) | ((rs["J"][feas] == kth) & (samp[feas] >= top[-1])) | in_top[feas])
    # the sampled feasible fraction agrees with n_feas (binomial, 6 sigma)
    f = g["n_feas"] / inst.space_size
    sd = np.sqrt(f * (1 - f) / len(samp))
    assert abs(feas.mean() - f) <= 6 * sd + 1e-3
    # the nearest competitors: every configuration one option away from a
    # top-64 member, and two options away from one of the best four (the
    # oracle on each)
    K = [int(k) for k in inst.n_options]
    strides = [int(np.prod(K[i + 1:])) for i in range(len(K))]

    def digits(x):
        return [(int(x) // strides[i]) % K[i] for i in range(len(K))]

    near = set()
    for x in top:
        d = digits(x)
        for i in range(len(K)):
            for o in range(K[i]):
                if o != d[i]:
                    near.add(int(x) + (o - d[i]) * strides[i])
    for x in top[:4]:
        d0 = digits(x)
        for i in range(len(K)):
            for j in range(i + 1, len(K)):
                for oi in range(K[i]):
                    for oj in range(K[j]):
                        if oi != d0[i] and oj != d0[j]:
                            near.add(int(x) + (oi - d0[i]) * strides[i] + (oj - d0[j]) * strides[j])
    near = np.array(sorted(near - set(int(t) for t in top)), dtype=np.uint64)
    rn = orc.Problem(inst).eval_list(near, inst.sla, inst.omega)
    fn = (rn["flags"] & 4) != 0
    print(f"[bf16] {len(near)} neighbours of the top-64, {int(fn.sum())} feasible", flush=True)
    assert fn.sum() > 0
    assert np.all((rn["J"][fn] < kth) | ((rn["J"][fn] == kth) & (near[fn] > top[-1])))


def _fingerprint(inst) -> str:
    h = hashlib.sha256()
    for a in (inst.n_options, inst.features, inst.agg_cols, inst.weights, inst.sla, inst.omega):
        h.update(np.ascontiguousarray(a).tobytes())
    h.update(np.float32(inst.vram_cap).tobytes())
    return h.hexdigest()[:16]


def test_bf16_n8_oracle_chunks(mf):
    # 64 chunks of 2^18 consecutive configurations of the N=8 workload (the
    # head, across the 2^31 midpoint, the tail and seeded offsets), each run
    # through the oracle in full when the golden file was written: counts,
    # the top-64 with canonical J, and every configuration's mask bits (as a
    # SHA-256 over the chunk's flag bytes)
    path = os.path.join(GOLDEN, "cfg4_s0_chunks.json")
    rec = json.load(open(path))
    inst = synth.cfg4(rec["seed"])
    assert _fingerprint(inst) == rec["fingerprint"], "the generator changed since the golden file was written"
    p = mf.Problem(inst)
    assert len(rec["chunks"]) >= 64
    for c in rec["chunks"]:
        lo, hi = c["lo"], c["hi"]
        print(f"[bf16] oracle chunk [{lo}, {hi})", flush=True)
        g = p.search(inst.sla, inst.omega, k=rec["k"], lo=lo, hi=hi, dump=True)
        assert g["n_vram"] == c["n_vram"] and g["n_feas"] == c["n_feas"], (lo, g["n_feas"], c["n_feas"])
        assert [int(x) for x in g["top_idx"]] == c["top_idx"], lo
        assert [float(x).hex() for x in g["top_J"]] == c["top_J"], lo
        flags = (g["mask"].cpu().numpy() & 7).astype(np.uint8)
        assert hashlib.sha256(flags.tobytes()).hexdigest() == c["flags_sha256"], lo


def test_bf16_topk_fallback_on_exact_ties(mf, orc):
    # throughput independent of the configuration: every feasible
    # configuration ties at J = N, more than the fast list holds
    inst = synth.make_instance([12, 11, 10], 8, 4, 64, 64, seed=4, vram_quantile=0.7, sla_range=(0.2, 1.0),
                               dtype="bf16")
    for i in range(inst.n_models):
        W1, b1, W2, b2, W3, b3 = inst.model_weights(i)
        W3[1, :] = 0.0
        b3[1] = 1.0
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=64)
    assert r["n_feas"] > 128
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=64)
    assert g["n_topk_collect"] > 0
    assert g["n_feas"] == r["n_feas"]
    assert list(g["top_idx"]) == list(r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_bf16_degenerate_ranges(mf, orc):
    inst = synth.cfg4(2)
    p = mf.Problem(inst)
    g = p.search(inst.sla, inst.omega, k=64, lo=1000, hi=1000)
    assert g["n_eval"] == 0 and g["n_feas"] == 0 and len(g["top_idx"]) == 0
    for lo in (0, 12_345_678, inst.space_size - 1):
        r = orc.Problem(inst).search(inst.sla, inst.omega, k=3, lo=lo, hi=lo + 1)
        g = p.search(inst.sla, inst.omega, k=3, lo=lo, hi=lo + 1)
        assert g["n_feas"] == r["n_feas"] and g["n_vram"] == r["n_vram"]
        assert list(g["top_idx"]) == list(r["top_idx"])
        assert g["top_J"].tobytes() == r["top_J"].tobytes()


def test_bf16_range_splits_when_certification_list_fills(mf, orc):
    # model 0's latency is the constant 0.25 and its bound is exactly 0.25:
    # every configuration sits on the (inclusive) boundary, so every one is
    # certified, and a 4-entry certification list forces many range splits
    inst = synth.make_instance([9, 8, 7, 6], 8, 4, 64, 64, seed=21, vram_quantile=0.8, sla_range=(0.2, 1.0),
                               dtype="bf16")
    W1, b1, W2, b2, W3, b3 = inst.model_weights(0)
    W3[0, :] = 0.0
    b3[0] = 0.25
    inst.sla[0] = 0.25
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=16)
    assert r["n_feas"] > 0
    g0 = mf.Problem(inst).search(inst.sla, inst.omega, k=16)
    assert g0["n_flagged"] >= r["n_feas"]
    g = mf.Problem(inst).search(inst.sla, inst.omega, k=16, worklist_cap=4)
    assert g["n_splits"] > 0
    assert g["n_feas"] == r["n_feas"] and g["n_vram"] == r["n_vram"]
    assert list(g["top_idx"]) == list(r["top_idx"])
    assert g["top_J"].tobytes() == r["top_J"].tobytes()
