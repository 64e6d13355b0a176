"""Pins of the oracle's subspace overlap score (Sec. 3, T^6 recovery score).

The score is pinned by facts independent of its formula: a span compared
with itself (or with any invertible mix of it, shifted) scores 1; centred
orthogonal spans score 0; spans sharing one of two directions score 1/2;
for single columns the score is the squared Pearson correlation (numpy's
corrcoef); and the score is symmetric in its two arguments.
"""
import numpy as np
import pytest

from oracle import diagnostics as od


def centred_orthonormal(n, k, seed):
    rng = np.random.default_rng(seed)
    Z = rng.normal(size=(n, k))
    Z -= Z.mean(0)
    Q, _ = np.linalg.qr(Z)
    return Q


def test_same_span_any_basis_and_shift_scores_one():
    rng = np.random.default_rng(0)
    A = rng.normal(size=(500, 2))
    M = np.array([[2.0, -1.0], [0.5, 3.0]])
    B = A @ M + np.array([4.0, -7.0])
    assert od.rv_overlap(A, B) == pytest.approx(1.0, abs=1e-12)
    assert od.rv_overlap(A, A) == pytest.approx(1.0, abs=1e-12)


def test_orthogonal_centred_spans_score_zero():
    Q = centred_orthonormal(400, 4, 1)
    assert od.rv_overlap(Q[:, :2], Q[:, 2:]) == pytest.approx(0.0, abs=1e-12)


def test_one_shared_direction_scores_half():
    Q = centred_orthonormal(300, 3, 2)
    A = Q[:, [0, 1]]
    B = Q[:, [0, 2]]
    assert od.rv_overlap(A, B) == pytest.approx(0.5, abs=1e-12)


def test_single_columns_give_squared_correlation():
    rng = np.random.default_rng(3)
    x = rng.normal(size=1000)
    y = 0.3 * x + rng.normal(size=1000)
    r = np.corrcoef(x, y)[0, 1]
    assert od.rv_overlap(x, y) == pytest.approx(r * r, rel=1e-12)


def test_symmetric_and_bounded():
    rng = np.random.default_rng(4)
    A = rng.normal(size=(200, 2))
    B = A + 0.7 * rng.normal(size=(200, 2))
    s = od.rv_overlap(A, B)
    assert s == pytest.approx(od.rv_overlap(B, A), rel=1e-12)
    assert 0.0 < s < 1.0


def test_circle_harmonic_recovered_exactly():
    # the score the paper applies: (cos t, sin t) of a circle against any
    # rotated, rescaled copy of itself is 1
    t = np.linspace(0, 2 * np.pi, 360, endpoint=False)
    B = np.stack([np.cos(t), np.sin(t)], 1)
    c, s = np.cos(0.7), np.sin(0.7)
    A = B @ np.array([[c, -s], [s, c]]) * 3.0
    assert od.rv_overlap(A, B) == pytest.approx(1.0, abs=1e-12)
