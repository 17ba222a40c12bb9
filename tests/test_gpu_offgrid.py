"""GPU parity on inputs off the 2^-14 grid (the feature values real profiling
tables would carry), against the CPU oracle, through the C ABI.

On the generator's default grid every fp32 aggregate sum is exact in any
order; off it, nearly every configuration's aggregate rounds, so these cases
check that every kernel forms the aggregate as the definition does (fp32 adds
in model order from zero), that the fast path's error bounds cover the
rounding of the centred aggregate a - c, and that the VRAM cap and latency
decisions are taken on those values.  Bars as in the on-grid tests: masks,
counts, top-k indices and canonical J bit-exact; fast predictions within
1e-5 (fp32) / 2e-2 (bf16, and 1e-4 by design) of the oracle.
"""
import numpy as np
import pytest

from paper_2609_02109_amd import synth
from test_gpu_fixed_state import fixed_parity
from test_gpu_ga import run_both
from test_gpu_search import check_predictions, run_range_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_02109_amd import mf as mfmod
    return mfmod


def off_grid(n_options, n_local, n_agg, hidden, seed, **kw):
    inst = synth.make_instance(n_options, n_local, n_agg, hidden, hidden, seed=seed, quantise=False, **kw)
    cols = inst.features[:, 3:].astype(np.float64)
    assert np.any(cols * 2 ** 14 != np.round(cols * 2 ** 14)), "the instance should be off the grid"
    return inst


def assert_inexact(orc, inst, lo, hi):
    r = orc.Problem(inst).search(inst.sla, inst.omega, k=1, lo=lo, hi=hi)
    assert r["n_inexact_agg"] > (hi - lo) // 2, "most aggregates should round in fp32"


@pytest.mark.parametrize("seed", [0, 1])
def test_offgrid_n5_full_space(mf, orc, seed):
    inst = off_grid([12, 12, 9, 9, 9], 8, 4, 32, seed, vram_quantile=0.75, top_k=16)
    assert_inexact(orc, inst, 0, inst.space_size)
    run_range_parity(mf, orc, inst, 0, inst.space_size, 16)


def test_offgrid_n5_tight_bounds(mf, orc):
    # latency bounds inside the prediction spread: many decisions go to the
    # canonical re-evaluation, which must see the same rounded aggregate
    inst = off_grid([12, 12, 9, 9, 9], 8, 4, 32, 5, vram_quantile=0.75, sla_range=(-0.15, 0.15), top_k=16)
    g, r = run_range_parity(mf, orc, inst, 0, inst.space_size, 16)
    assert g["n_flagged"] > 0 and 0 < r["n_feas"] < r["n_vram"]


def test_offgrid_n6_ranges(mf, orc):
    inst = off_grid([24] * 6, 16, 6, 64, 0, vram_cap=200.0)
    assert_inexact(orc, inst, 0, 1 << 14)
    run_range_parity(mf, orc, inst, 0, 1 << 17, 4)
    n = inst.space_size
    run_range_parity(mf, orc, inst, n // 2 - 40_001, n // 2 + 60_000, 8)


def test_offgrid_n6_vram_cap_at_a_rounded_sum(mf, orc):
    # the cap equal to one configuration's fp32 VRAM sum: the inclusive
    # comparison at the cap sees exactly the rounded model-order sum
    inst = off_grid([24] * 6, 16, 6, 64, 3, vram_cap=200.0)
    a, _ = orc.Problem(inst).aggregate(orc.Problem(inst).decode(777_777))
    inst.vram_cap = float(a[inst.vram_slot])
    g, r = run_range_parity(mf, orc, inst, 700_000, 900_000, 4)
    assert g["mask"][77_777].item() & 1


def test_offgrid_n8_bf16_ranges(mf, orc):
    inst = off_grid([16] * 8, 32, 8, 256, 0, vram_cap=288.0, dtype="bf16", top_k=64)
    assert_inexact(orc, inst, 0, 1 << 12)
    g, r = run_range_parity(mf, orc, inst, (1 << 31) - 20_000, (1 << 31) + 30_001, 64, tol=2e-2)
    check_predictions(g["pred"].cpu().numpy(), r["pred"], tol=1e-4)


@pytest.mark.parametrize("n_options,n_local,n_agg,hidden,dtype,k", [
    ([12, 12, 9, 9, 9], 8, 4, 32, "f32", 16),
    ([9, 7, 8, 6], 16, 6, 64, "bf16", 8),
])
def test_offgrid_fixed_state_full_space(mf, orc, n_options, n_local, n_agg, hidden, dtype, k):
    inst = off_grid(n_options, n_local, n_agg, hidden, 2, vram_quantile=0.7, dtype=dtype)
    fixed_parity(mf, orc, inst, synth.make_state(inst, 2), 0, inst.space_size, k)


def test_offgrid_ga(mf, orc):
    # the GA's feasible list, repair and fitness on rounded aggregates: whole
    # trajectories identical to the oracle's replay
    inst = off_grid([12, 12, 9, 9, 9], 8, 4, 32, 4, vram_quantile=0.75)
    sc = synth.ga_scenarios(5, 4, seed=4)
    run_both(mf, orc, inst, sc.sla, sc.omega, pop=256, gens=20, seed=11)
    run_both(mf, orc, inst, sc.sla[:1], sc.omega[:1], pop=100, gens=30, p_mut=0.1, seed=2)
