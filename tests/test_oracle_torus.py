"""Pins of the grid-torus closed form, Nystrom and diagnostics (CPU only).

* Circulant eigenvalues agree with numpy's FFT of the first row.
* The Kronecker-circulant spectrum and product agree with the dense oracle.
* Continuum limit: on a fine grid lambda(m) / lambda(0) -> I_m(2 beta R^2) /
  I_0(2 beta R^2) (trapezoidal rule for the Bessel integral; scipy).
* Multiplicities on a square flat 2-torus follow the count of integer
  vectors with m1^2 + m2^2 = shell: 1, 4, 4, 4, 8.
* The paper's T^6 radii (golden fixture) order the first-harmonic doublets
  as the Laplace-Beltrami closed form m^2 / R^2 says, and in the heat-kernel
  regime 4 beta (-log lambda_1/lambda_0) approaches 1 / R^2.
* Nystrom extension onto the same points returns the eigenvectors.
* Precision table and Perron wall constants match the golden fixture.
"""
import math

import numpy as np
import pytest
import scipy.special

from conftest import read_golden
from oracle import diagnostics as od
from oracle import eig as oe
from oracle import kernel as ok
from oracle import normalise as on
from oracle import nystrom as ony
from oracle import torus_grid as tg


def grid_points(counts, radii=None):
    # independent construction of the grid (mirrors the point order of the
    # closed form: first axis slowest)
    R = np.ones(len(counts)) if radii is None else np.asarray(radii, float)
    idx = np.indices(counts).reshape(len(counts), -1).T
    th = 2 * np.pi * idx / np.asarray(counts)[None, :]
    X = np.empty((idx.shape[0], 2 * len(counts)))
    X[:, 0::2] = R * np.cos(th)
    X[:, 1::2] = R * np.sin(th)
    return X


@pytest.mark.parametrize("n,R,beta", [(7, 1.0, 0.5), (16, 1.3, 2.0), (33, 0.8, 8.0)])
def test_circulant_eigs_match_fft(n, R, beta):
    c = tg.circulant_first_row(n, R, beta)
    ref = np.fft.fft(c).real
    np.testing.assert_allclose(tg.circulant_eigs(n, R, beta), ref, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("counts,radii,beta", [((8, 6), None, 1.5), ((5, 4, 3), (1.0, 1.2, 0.7), 0.8)])
def test_closed_form_matches_dense(counts, radii, beta):
    X = grid_points(counts, radii)
    K = ok.gaussian_kernel(X, None, beta)
    ev_dense = np.sort(np.linalg.eigvalsh(K))[::-1]
    ev_cf = np.sort(tg.kernel_eigs(counts, beta, radii))[::-1]
    np.testing.assert_allclose(ev_cf, ev_dense, atol=1e-11)
    q = K.sum(1)
    np.testing.assert_allclose(q, tg.degree(counts, beta, radii), rtol=1e-12)
    M, _ = on.operator_M(X, beta, 0.5, K=K)
    np.testing.assert_allclose(tg.operator_eigs(counts, beta, radii),
                               np.sort(np.linalg.eigvalsh(M))[::-1], atol=1e-12)
    V = np.random.default_rng(2).normal(size=(X.shape[0], 3))
    np.testing.assert_allclose(tg.kernel_apply(counts, beta, V, radii), K @ V, rtol=1e-11, atol=1e-12)
    # Fourier modes are eigenvectors
    v = tg.fourier_mode(counts, (1,) + (0,) * (len(counts) - 1))
    lam = tg.circulant_eigs(counts[0], 1.0 if radii is None else radii[0], beta)[1]
    lam *= np.prod([tg.circulant_eigs(n, 1.0 if radii is None else r, beta)[0]
                    for n, r in zip(counts[1:], (radii or (1.0,) * len(counts))[1:])])
    np.testing.assert_allclose(K @ v, lam * v, atol=1e-11)


@pytest.mark.parametrize("R,beta", [(1.0, 0.5), (1.5, 2.0), (0.9, 6.0)])
def test_bessel_continuum_limit(R, beta):
    n = 256
    lam = tg.circulant_eigs(n, R, beta)
    x = 2 * beta * R * R
    for m in range(5):
        ref = scipy.special.ive(m, x) / scipy.special.ive(0, x)
        assert lam[m] / lam[0] == pytest.approx(ref, rel=1e-10)
    # absolute: lambda(0) = n e^{-x} I_0(x)
    assert lam[0] == pytest.approx(n * scipy.special.ive(0, x), rel=1e-10)


def test_square_torus_multiplicities():
    counts = (12, 12)
    X = grid_points(counts)
    M, _ = on.operator_M(X, 0.9, 0.5)
    lam = np.sort(np.linalg.eigvalsh(M))[::-1]
    # group into clusters
    groups = []
    i = 0
    while len(groups) < 5:
        j = i
        while j + 1 < lam.size and abs(lam[j + 1] - lam[i]) < 1e-10:
            j += 1
        groups.append(j - i + 1)
        i = j + 1
    assert groups == [1, 4, 4, 4, 8]


def test_t6_radii_order_first_harmonic_doublets():
    g = read_golden("t6_torus_spectrum.txt")
    R = np.array([float(v) for v in g["radii"]])
    lead = int(g["leading_doublet_circle"][0])
    assert 1.0 / R.min() ** 2 == pytest.approx(float(g["largest_first_harmonic"][0]), abs=5e-3)
    assert 4.0 / R.max() ** 2 == pytest.approx(float(g["smallest_second_harmonic"][0]), abs=5e-4)
    assert 4.0 / R.max() ** 2 - 1.0 / R.min() ** 2 == pytest.approx(float(g["band_gap"][0]), abs=5e-3)
    n = 128
    beta = 40.0
    first = []
    for r in R:
        lam = tg.circulant_eigs(n, r, beta)
        first.append(lam[1] / lam[0])
        # doublet: m = 1 and m = n-1 are equal
        assert lam[1] == pytest.approx(lam[n - 1], rel=1e-12)
    first = np.array(first)
    assert int(np.argmax(first)) == lead
    assert np.all(np.diff(first) > 0)  # larger circle, larger eigenvalue
    heat = -4 * beta * np.log(first)
    np.testing.assert_allclose(heat, 1.0 / R ** 2, rtol=0.02)
    # second harmonic of the largest circle lies below every first harmonic
    lam = tg.circulant_eigs(n, R.max(), beta)
    assert lam[2] / lam[0] < first.min()


def test_nystrom_same_points_is_identity():
    X = np.random.default_rng(4).normal(size=(70, 3))
    sp = oe.spectrum(X, 0.9, 0.5, 5)
    ext = ony.nystrom_extend(X, X, 0.9, 0.5, sp.psi, sp.evals, q_old=sp.norm.q)
    np.testing.assert_allclose(ext, sp.psi, rtol=1e-9, atol=1e-12)


def test_nystrom_converges_on_nested_samples():
    # extend from the first 400 points to all 1600 points of a circle and
    # compare with the eigenvectors solved on all 1600: small angle
    rng = np.random.default_rng(9)
    th = rng.uniform(0, 2 * np.pi, 1600)
    X = np.stack([np.cos(th), np.sin(th)], 1)
    beta = 2.0
    small = oe.spectrum(X[:400], beta, 0.5, 3)
    ext = ony.nystrom_extend(X[:400], X, beta, 0.5, small.psi, small.evals)
    full = oe.spectrum(X, beta, 0.5, 3)
    ang = od.principal_angles(ext[:, :3], full.psi[:, :3])
    assert ang.max() < 0.05


def test_precision_table_and_wall():
    g = read_golden("precision_eta.txt")
    for name, val in g["eta"]:
        assert od.ETA[name] == pytest.approx(float(val), rel=1e-12)
    assert od.KAPPA_P == float(g["kappa_P"][0])
    assert od.P_EXPONENT == int(g["p"][0])
    # two-point Perron gap 2e/(1+e): wall crossing is decided by it
    for beta, expect in [(0.1, True), (16.0, False)]:
        X = np.array([[0.0, 0.0], [1.0, 0.0]])
        sp = oe.spectrum(X, beta, 0.5, 2)
        e = math.exp(-beta)
        assert od.perron_gap(sp.evals) == pytest.approx(2 * e / (1 + e), rel=1e-6)
        assert od.wall_admissible(od.perron_gap(sp.evals), "fp32") == expect
    assert od.v_mach(1e-6, "fp32") == pytest.approx(1.0)


def test_principal_angles_known_cases():
    A = np.eye(4)[:, :2]
    assert od.principal_angles(A, A).max() < 1e-12
    B = np.eye(4)[:, 2:]
    np.testing.assert_allclose(od.principal_angles(A, B), [np.pi / 2] * 2)
    t = 0.3
    C = np.array([[1, 0], [0, math.cos(t)], [0, math.sin(t)], [0, 0]])
    np.testing.assert_allclose(np.sort(od.principal_angles(A, C)), [0.0, t], atol=1e-12)
