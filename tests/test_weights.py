"""Folding an inference-mode batch norm into the preceding linear layer: the
folded layer reproduces torch's Linear -> BatchNorm1d (eval) in float64 to
rounding, and the packed row has the layout the library reads."""
import numpy as np
import torch

from paper_2609_02109_amd import synth
from paper_2609_02109_amd.weights import fold_batchnorm, pack_model


def test_fold_batchnorm_matches_torch():
    rng = np.random.default_rng(0)
    nin, h = 12, 64
    lin = torch.nn.Linear(nin, h).double()
    bn = torch.nn.BatchNorm1d(h, eps=1e-5).double()
    with torch.no_grad():
        bn.weight.copy_(torch.from_numpy(rng.uniform(0.5, 2.0, h)))
        bn.bias.copy_(torch.from_numpy(rng.normal(0, 0.3, h)))
        bn.running_mean.copy_(torch.from_numpy(rng.normal(0, 0.5, h)))
        bn.running_var.copy_(torch.from_numpy(rng.uniform(0.2, 3.0, h)))
    bn.eval()
    x = torch.from_numpy(rng.normal(0, 1, (256, nin)))
    ref = bn(lin(x)).detach().numpy()
    Wf, bf = fold_batchnorm(lin.weight.detach().numpy(), lin.bias.detach().numpy(), bn.weight.detach().numpy(),
                            bn.bias.detach().numpy(), bn.running_mean.numpy(), bn.running_var.numpy(), 1e-5)
    got = x.numpy() @ Wf.astype(np.float64).T + bf.astype(np.float64)
    # the folded weights are rounded to fp32 once: agreement to fp32 rounding
    assert np.max(np.abs(got - ref) / (np.abs(ref) + 1.0)) < 1e-5


def test_pack_model_layout():
    inst = synth.make_instance([3, 4], 8, 4, 64, 32, seed=1, vram_cap=80.0)
    parts = inst.model_weights(1)
    row = pack_model(*parts)
    assert row.tobytes() == inst.weights[1].tobytes()
