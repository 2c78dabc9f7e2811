"""Pins of the fp64 projection-product oracle (CPU): a scalar triple loop,
central finite differences of L = sum(Y * dY) (calculus ties the two gradients
to the forward), and the transpose identity."""
import itertools

import numpy as np
import pytest

import oracle


def _loop_matmul(a, b):
    M, K = a.shape
    N = b.shape[1]
    out = np.zeros((M, N))
    for i in range(M):
        for j in range(N):
            s = 0.0
            for t in range(K):
                s += float(a[i, t]) * float(b[t, j])
            out[i, j] = s
    return out


@pytest.mark.parametrize("M,K,N", [(1, 1, 1), (3, 5, 2), (4, 7, 6)])
def test_proj_matches_scalar_loops(M, K, N):
    rng = np.random.default_rng(M * 100 + K * 10 + N)
    x, w, dy = rng.standard_normal((M, K)), rng.standard_normal((K, N)), rng.standard_normal((M, N))
    np.testing.assert_allclose(oracle.proj_fwd(x, w), _loop_matmul(x, w), rtol=0, atol=1e-13)
    # dX[i, t] = sum_j dY[i, j] W[t, j];  dW[t, j] = sum_i X[i, t] dY[i, j]
    dx = np.array([[sum(dy[i, j] * w[t, j] for j in range(N)) for t in range(K)] for i in range(M)])
    dw = np.array([[sum(x[i, t] * dy[i, j] for i in range(M)) for j in range(N)] for t in range(K)])
    np.testing.assert_allclose(oracle.proj_bwd_data(dy, w), dx, rtol=0, atol=1e-13)
    np.testing.assert_allclose(oracle.proj_bwd_weight(x, dy), dw, rtol=0, atol=1e-13)


def test_proj_gradients_match_central_differences():
    rng = np.random.default_rng(5)
    M, K, N = 3, 4, 5
    x, w, dy = rng.standard_normal((M, K)), rng.standard_normal((K, N)), rng.standard_normal((M, N))
    loss = lambda x_, w_: float(np.sum(oracle.proj_fwd(x_, w_) * dy))
    h = 1e-6
    for which, g in ((0, oracle.proj_bwd_data(dy, w)), (1, oracle.proj_bwd_weight(x, dy))):
        base = [x, w]
        fd = np.zeros_like(base[which])
        for idx in itertools.product(*(range(n) for n in base[which].shape)):
            plus = [a.copy() for a in base]
            minus = [a.copy() for a in base]
            plus[which][idx] += h
            minus[which][idx] -= h
            fd[idx] = (loss(*plus) - loss(*minus)) / (2 * h)
        np.testing.assert_allclose(g, fd, rtol=0, atol=1e-7)


def test_weight_gradient_transpose_identity():
    rng = np.random.default_rng(9)
    x, dy = rng.standard_normal((17, 6)), rng.standard_normal((17, 9))
    np.testing.assert_allclose(oracle.proj_bwd_weight(x, dy).T, dy.T @ x, rtol=0, atol=1e-12)
