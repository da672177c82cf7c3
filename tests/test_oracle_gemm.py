"""Pins for the FP64 linear-layer oracle (forward and straight-through backward).

Checked against pure-Python triple loops on tiny shapes (non-square, so a transposed
operand cannot pass), the identity-input closed form, and the gradient decomposition
dW(W4A4) = dO A^T + dO eps_A^T of Eq. activation-gradient-error.
"""
import numpy as np

import oracle
from tests.helpers import bf16_to_f64
from workloads import normal_bf16


def _loops_fwd(a, w):
    M, K = a.shape
    N = w.shape[0]
    return [[sum(a[i][k] * w[j][k] for k in range(K)) for j in range(N)] for i in range(M)]


def _loops_dx(dy, w):
    M, N = dy.shape
    K = w.shape[1]
    return [[sum(dy[i][n] * w[n][k] for n in range(N)) for k in range(K)] for i in range(M)]


def _loops_dw(dy, a):
    M, N = dy.shape
    K = a.shape[1]
    return [[sum(dy[m][n] * a[m][k] for m in range(M)) for k in range(K)] for n in range(N)]


def test_linear_oracle_matches_triple_loops():
    rng = np.random.default_rng(0)
    M, N, K = 5, 7, 32
    a = normal_bf16(rng, (M, K))
    w = normal_bf16(rng, (N, K), 0.02)
    dy = normal_bf16(rng, (M, N))
    A, Wf, D = bf16_to_f64(a).tolist(), bf16_to_f64(w).tolist(), bf16_to_f64(dy).tolist()
    A, Wf, D = np.array(A), np.array(Wf), np.array(D)
    np.testing.assert_allclose(oracle.linear_fwd(a, w), _loops_fwd(A, Wf), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(oracle.linear_dx(dy, w), _loops_dx(D, Wf), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(oracle.linear_dw(dy, a), _loops_dw(D, A), rtol=1e-13, atol=1e-15)
    assert oracle.linear_fwd(a, w).shape == (M, N)
    assert oracle.linear_dx(dy, w).shape == (M, K)
    assert oracle.linear_dw(dy, a).shape == (N, K)


def test_identity_input_returns_quantized_weight_rows():
    rng = np.random.default_rng(1)
    K, N = 64, 48
    w = normal_bf16(rng, (N, K), 0.02)
    what = oracle.fakequant(w, "nvfp4")
    eye = np.zeros((K, K), np.uint16)
    eye[np.arange(K), np.arange(K)] = 0x3F80
    y = oracle.linear_fwd(eye, what)
    np.testing.assert_array_equal(y, bf16_to_f64(what).T)


def test_activation_gradient_decomposition():
    rng = np.random.default_rng(2)
    M, N, K = 40, 24, 64
    a = normal_bf16(rng, (M, K))
    dy = normal_bf16(rng, (M, N))
    ahat = oracle.fakequant(a, "mxfp4")
    eps = bf16_to_f64(ahat) - bf16_to_f64(a)
    lhs = oracle.linear_dw(dy, ahat) - oracle.linear_dw(dy, a)
    rhs = bf16_to_f64(dy).T @ eps
    np.testing.assert_allclose(lhs, rhs, rtol=1e-10, atol=1e-12)
    assert np.abs(rhs).max() > 0


def test_sampled_entries_match_full_product():
    rng = np.random.default_rng(3)
    a = normal_bf16(rng, (33, 96))
    w = normal_bf16(rng, (17, 96), 0.02)
    full = oracle.linear_fwd(a, w)
    ii = rng.integers(0, 33, 50)
    jj = rng.integers(0, 17, 50)
    np.testing.assert_allclose(oracle.dot_rows(a, ii, w, jj), full[ii, jj], rtol=1e-14, atol=1e-16)
