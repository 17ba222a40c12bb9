"""GPU parity on a seeded sweep of random instance shapes (through the C ABI).

Each case draws the number of models, their option counts, the feature and
aggregate widths, the hidden width, the weight dtype, the VRAM cap quantile,
the latency bounds, k and a sub-range of the joint space from its own seed,
then compares the whole exhaustive search over that range (masks, counts,
top-k, canonical J, fast-path predictions) with the oracle, to the same bars
as the fixed-shape tests.  The space is sized so that the oracle finishes in
about a second per case.
"""
import numpy as np
import pytest

from paper_2609_02109_amd import synth
from test_gpu_search import check_predictions, run_range_parity

pytestmark = pytest.mark.gpu

# oracle work bound per case: configurations x models x hidden^2
WORK = 4e9


@pytest.fixture(scope="module")
def mf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_02109_amd import mf as mfmod
    return mfmod


def draw_case(seed):
    rng = np.random.default_rng(1000 + seed)
    bf16 = seed % 2 == 1
    H = int(rng.choice([64, 128, 256] if bf16 else [32, 64]))
    A = int(rng.choice([2, 4, 6, 8]))
    L = int(rng.choice([8, 12, 16, 24, 32]))
    N = int(rng.integers(1, 9))
    cap = max(2, int(WORK / (N * H * H)))
    K = []
    for i in range(N):
        room = cap // max(1, int(np.prod(K)) if K else 1)
        K.append(int(rng.integers(1, max(2, min(13, room + 1)))))
    lo_q, hi_q = sorted(rng.uniform(-0.3, 1.0, 2))
    return dict(n_options=K, n_local=L, n_agg=A, hidden=H, dtype="bf16" if bf16 else "f32",
                vram_quantile=float(rng.uniform(0.3, 0.95)), sla_range=(float(lo_q), float(hi_q) + 0.05),
                k=int(rng.integers(1, 65)), range_seed=int(rng.integers(0, 2 ** 31)))


@pytest.mark.parametrize("seed", range(32))
def test_random_shape(mf, orc, seed):
    c = draw_case(seed)
    inst = synth.make_instance(c["n_options"], c["n_local"], c["n_agg"], c["hidden"], c["hidden"], seed=seed,
                               vram_quantile=c["vram_quantile"], sla_range=c["sla_range"], dtype=c["dtype"])
    n = inst.space_size
    rng = np.random.default_rng(c["range_seed"])
    if seed % 4 == 0 or n < 4:
        lo, hi = 0, n
    else:
        lo = int(rng.integers(0, n // 2))
        hi = int(rng.integers(lo + 1, n + 1))
    print(f"[random] seed={seed} K={c['n_options']} L={c['n_local']} A={c['n_agg']} H={c['hidden']} "
          f"{c['dtype']} k={c['k']} range=[{lo},{hi})", flush=True)
    tol = 2e-2 if c["dtype"] == "bf16" else 1e-5
    g, r = run_range_parity(mf, orc, inst, lo, hi, c["k"], tol=tol)
    if c["dtype"] == "bf16":
        check_predictions(g["pred"].cpu().numpy(), r["pred"], tol=1e-4)
    assert len(g["top_idx"]) == min(c["k"], r["n_feas"])
