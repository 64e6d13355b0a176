"""Pins of the oracle's normalisation and dense eigensolve (CPU only).

Properties fixed by Sec. 2.1: P is row-stochastic; M = diag(d)^1/2 P
diag(d)^-1/2 so M sqrt(d) = sqrt(d) and lambda_0 = 1; M and P share their
spectrum; spec(M) lies in [0, 1]; alpha = 0 gives D^-1/2 K D^-1/2.
Sec. 2.3: S_off = sum_{i != j} K_ij.  The two-point problem has the closed
form spec(M) = {1, (1 - e) / (1 + e)}, e = exp(-beta ||x1 - x2||^2), for any
alpha (q is constant, so M = K / (1 + e)).
"""
import math

import numpy as np
import pytest

from oracle import eig as oe
from oracle import kernel as ok
from oracle import normalise as on


def _pts(n=60, d=3, seed=11):
    return np.random.default_rng(seed).normal(size=(n, d))


@pytest.mark.parametrize("alpha", [0.0, 0.5, 1.0])
def test_P_row_stochastic_and_similar_to_M(alpha):
    X = _pts()
    P = on.operator_P(X, 0.8, alpha)
    np.testing.assert_allclose(P.sum(axis=1), np.ones(60), rtol=1e-13)
    M, nrm = on.operator_M(X, 0.8, alpha)
    np.testing.assert_allclose(M, M.T, rtol=0, atol=1e-15)
    # M = D^1/2 P D^-1/2
    sd = np.sqrt(nrm.d)
    np.testing.assert_allclose(M, sd[:, None] * P / sd[None, :], rtol=1e-12, atol=1e-15)
    # shared spectrum
    lp = np.sort(np.linalg.eigvals(P).real)[::-1]
    lm = np.sort(np.linalg.eigvalsh(M))[::-1]
    np.testing.assert_allclose(lp, lm, atol=1e-11)


@pytest.mark.parametrize("alpha", [0.0, 0.5, 1.0])
def test_perron_vector_and_spectrum_range(alpha):
    X = _pts()
    M, nrm = on.operator_M(X, 1.7, alpha)
    sd = np.sqrt(nrm.d)
    np.testing.assert_allclose(M @ sd, sd, rtol=1e-12)
    lam = np.linalg.eigvalsh(M)
    assert lam.max() == pytest.approx(1.0, abs=1e-12)
    assert lam.min() >= -1e-12


def test_alpha_zero_reduces_to_symmetric_laplacian_form():
    X = _pts()
    K = ok.gaussian_kernel(X, None, 0.6)
    q = K.sum(1)
    M, nrm = on.operator_M(X, 0.6, 0.0)
    np.testing.assert_allclose(nrm.s, q ** -0.5, rtol=1e-14)
    np.testing.assert_allclose(M, K / np.sqrt(np.outer(q, q)), rtol=1e-13)


def test_s_off_identity_and_matrix_free_normalisation():
    X = _pts(50, 4)
    K = ok.gaussian_kernel(X, None, 0.9)
    mask = ~np.eye(50, dtype=bool)
    ref = K[mask].sum()
    nrm = on.normalise(X, 0.9, 0.5, rows_block=13)
    assert nrm.s_off == pytest.approx(ref, rel=1e-13)
    _, dense = on.operator_M(X, 0.9, 0.5)
    for name in ("q", "w", "d", "s"):
        np.testing.assert_allclose(getattr(nrm, name), getattr(dense, name), rtol=1e-13)


@pytest.mark.parametrize("alpha", [0.0, 0.5, 1.0])
def test_two_point_closed_form(alpha):
    X = np.array([[0.3, -0.2, 1.0], [-0.5, 0.4, 0.1]])
    beta = 0.7
    h = float(np.sum((X[0] - X[1]) ** 2))
    e = math.exp(-beta * h)
    sp = oe.spectrum(X, beta, alpha, 2)
    np.testing.assert_allclose(sp.evals, [1.0, (1 - e) / (1 + e)], rtol=1e-14)


def test_markov_eigvecs_are_right_eigvecs_of_P():
    X = _pts(40, 2)
    sp = oe.spectrum(X, 1.1, 0.5, 6)
    P = on.operator_P(X, 1.1, 0.5)
    np.testing.assert_allclose(P @ sp.psi, sp.psi * sp.evals[None, :], atol=1e-11)
    # the Perron Markov vector is constant
    c = sp.psi[:, 0]
    np.testing.assert_allclose(c, np.full_like(c, c[0]), rtol=1e-10)


def test_top_eigenpairs_orders_and_sign_fix():
    A = np.diag([0.1, 0.9, 0.5, 1.0])
    w, V = oe.top_eigenpairs(A, 3)
    np.testing.assert_allclose(w, [1.0, 0.9, 0.5])
    np.testing.assert_allclose(np.abs(V[3, 0]), 1.0)
    S = oe.sign_fix(-V)
    assert np.all(S[np.argmax(np.abs(S), axis=0), np.arange(3)] > 0)
