"""Pins of the oracle's Gaussian affinity and products (CPU only).

Each check fixes the oracle to something other than itself: a hand-worked
value, an independent library routine (scipy cdist), or an exact property
of the kernel of Sec. 2.1 (symmetry, unit diagonal, positive
semidefiniteness, K(2 beta) = K(beta)^2 from Sec. 2.3, invariance under
translation / rotation / permutation, the beta = 0 rank-one limit).
"""
import math

import numpy as np
import pytest
import scipy.spatial.distance as ssd

from oracle import kernel as ok


def _pts(n=40, d=5, seed=3):
    return np.random.default_rng(seed).normal(size=(n, d))


def test_hand_worked_pair():
    # ||(0,0) - (1,2)||^2 = 1 + 4 = 5
    X = np.array([[0.0, 0.0], [1.0, 2.0]])
    K = ok.gaussian_kernel(X, None, 0.3)
    assert K[0, 1] == pytest.approx(math.exp(-1.5), rel=1e-15)
    assert K[0, 0] == 1.0 and K[1, 1] == 1.0
    # Y = K V by hand
    V = np.array([[2.0], [-1.0]])
    Y = ok.kernel_matmul(X, None, 0.3, V)
    e = math.exp(-1.5)
    assert Y[0, 0] == pytest.approx(2.0 - e, rel=1e-15)
    assert Y[1, 0] == pytest.approx(2.0 * e - 1.0, rel=1e-15)


def test_sq_distances_match_scipy_cdist():
    X = _pts(30, 7)
    Z = _pts(20, 7, seed=4)
    H = ok.sq_distances(X, Z)
    ref = ssd.cdist(X, Z, metric="sqeuclidean")
    np.testing.assert_allclose(H, ref, rtol=1e-13, atol=1e-13)


def test_symmetric_unit_diagonal_bounded():
    X = _pts()
    K = ok.gaussian_kernel(X, None, 0.7)
    np.testing.assert_array_equal(K, K.T)
    np.testing.assert_array_equal(np.diag(K), np.ones(X.shape[0]))
    assert np.all(K > 0) and np.all(K <= 1)


def test_positive_semidefinite():
    X = _pts(80, 3)
    K = ok.gaussian_kernel(X, None, 2.0)
    lam = np.linalg.eigvalsh(K)
    assert lam.min() >= -1e-12 * X.shape[0]


def test_dyadic_square_identity():
    # K(2 beta) = K(beta) elementwise squared (Sec. 2.3).
    X = _pts()
    K1 = ok.gaussian_kernel(X, None, 0.45)
    K2 = ok.gaussian_kernel(X, None, 0.9)
    np.testing.assert_allclose(K2, K1 * K1, rtol=1e-13, atol=0)


def test_translation_rotation_permutation():
    rng = np.random.default_rng(5)
    X = _pts(25, 4)
    K = ok.gaussian_kernel(X, None, 1.3)
    shift = rng.normal(size=(1, 4)) * 10
    np.testing.assert_allclose(ok.gaussian_kernel(X + shift, None, 1.3), K, rtol=1e-11, atol=1e-14)
    Q, _ = np.linalg.qr(rng.normal(size=(4, 4)))
    np.testing.assert_allclose(ok.gaussian_kernel(X @ Q, None, 1.3), K, rtol=1e-11, atol=1e-14)
    p = rng.permutation(25)
    np.testing.assert_array_equal(ok.gaussian_kernel(X[p], None, 1.3), K[np.ix_(p, p)])


def test_beta_zero_is_all_ones():
    X = _pts()
    np.testing.assert_array_equal(ok.gaussian_kernel(X, None, 0.0), np.ones((40, 40)))
    V = np.random.default_rng(0).normal(size=(40, 3))
    np.testing.assert_allclose(ok.kernel_matmul(X, None, 0.0, V), np.tile(V.sum(0), (40, 1)), rtol=1e-13)


def test_products_rows_rectangular_scaling():
    rng = np.random.default_rng(7)
    Xr = _pts(33, 6)
    Xc = _pts(21, 6, seed=8)
    V = rng.normal(size=(21, 5))
    sl = rng.uniform(0.5, 2.0, size=33)
    sr = rng.uniform(0.5, 2.0, size=21)
    Kd = ok.gaussian_kernel(Xr, Xc, 0.4)
    Y = ok.kernel_matmul(Xr, Xc, 0.4, V, sl=sl, sr=sr, block=7)
    # diag(sl) K diag(sr) V by explicit diagonal matrices
    ref = np.diag(sl) @ Kd @ np.diag(sr) @ V
    np.testing.assert_allclose(Y, ref, rtol=1e-13, atol=1e-15)
    rows = [0, 5, 32, 17]
    np.testing.assert_allclose(ok.kernel_matmul(Xr, Xc, 0.4, V, sl=sl, sr=sr, rows=rows), Y[rows], rtol=1e-14)
    # K(Xr, Xc)^T = K(Xc, Xr)
    np.testing.assert_array_equal(ok.gaussian_kernel(Xc, Xr, 0.4), Kd.T)
    # threads give the same rows
    np.testing.assert_array_equal(ok.kernel_matmul(Xr, Xc, 0.4, V, sl=sl, sr=sr, block=4, threads=3),
                                  ok.kernel_matmul(Xr, Xc, 0.4, V, sl=sl, sr=sr, block=4))
