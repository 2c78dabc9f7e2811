"""Projection matrix products of a fine-tuning step in float64 numpy (oracle;
test infrastructure only).

The linear layers around attention (the QKV and output projections, and the
LoRA A/B products of the paper's section 2.2 example) run on token-major
activations X [M tokens, K features] and a weight W [K, N]:
    forward          Y  = X W           (reduces over K)
    data gradient    dX = dY W^T        (reduces over N)
    weight gradient  dW = X^T dY        (reduces over the M tokens)
Section 4.1 classes matrix products as forward-tensor-dependent operators
whose gradients reduce along other axes than the forward (section 4.2: the
forward reduces along K, the gradients along N and M) -- the same stored
tensors are read along different dimensions.  These are the textbook
definitions written out with numpy's matrix product.

Pins (tests/test_oracle_proj.py): a scalar triple loop, central finite
differences of sum(Y * dY) with respect to X and W, and the transpose identity
dW^T = dY^T X.
"""
import numpy as np


def proj_fwd(x, w):
    """Y = X W: x (M, K), w (K, N) -> (M, N), float64."""
    return np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64)


def proj_bwd_data(dy, w):
    """dX = dY W^T: dy (M, N), w (K, N) -> (M, K), float64."""
    return np.asarray(dy, dtype=np.float64) @ np.asarray(w, dtype=np.float64).T


def proj_bwd_weight(x, dy):
    """dW = X^T dY: x (M, K), dy (M, N) -> (K, N), float64."""
    return np.asarray(x, dtype=np.float64).T @ np.asarray(dy, dtype=np.float64)
