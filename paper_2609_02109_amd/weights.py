"""Weight preparation for trained predictors (host side, before creation).

The paper's predictor (Section III-B) places batch normalisation after its
hidden linear layers.  At inference a batch-norm layer is the affine map
x -> gamma (x - mean) / sqrt(var + eps) + beta per unit, so it folds into the
preceding linear layer: W' = diag(s) W and b' = s (b - mean) + beta with
s = gamma / sqrt(var + eps).  Dropout is the identity at inference.  The
library's canonical semantics are defined on the weights it is given, so the
folded fp32 weights are what results are exact for.
"""
import numpy as np


def fold_batchnorm(W, b, gamma, beta, mean, var, eps=1e-5):
    """Fold an inference-mode batch norm that follows y = W x + b into (W', b'),
    computed in fp64 and rounded once to fp32."""
    W = np.asarray(W, np.float64)
    b = np.asarray(b, np.float64)
    s = np.asarray(gamma, np.float64) / np.sqrt(np.asarray(var, np.float64) + float(eps))
    Wf = W * s[:, None]
    bf = s * (b - np.asarray(mean, np.float64)) + np.asarray(beta, np.float64)
    return Wf.astype(np.float32), bf.astype(np.float32)


def pack_model(W1, b1, W2, b2, W3, b3):
    """One model's packed weight row in the layout mf_problem_create reads:
    W1[H1][L+A], b1[H1], W2[H2][H1], b2[H2], W3[2][H2], b3[2]."""
    return np.concatenate([np.asarray(x, np.float32).ravel() for x in (W1, b1, W2, b2, W3, b3)])
