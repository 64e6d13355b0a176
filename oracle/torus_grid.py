"""Closed-form Gaussian kernel on a regular grid of a flat torus, float64.

Test infrastructure.  A grid point has angles theta_a = 2 pi i_a / n_a and
is embedded as (R_a cos theta_a, R_a sin theta_a) for each axis a.  Its
squared distance to another grid point is

    sum_a 2 R_a^2 (1 - cos(theta_a - theta'_a)),

so the kernel of Sec. 2.1 (eq. kernel) factorises into a Kronecker product
of circulant matrices, K = C_1 (x) C_2 (x) ... with
C_a[i, j] = c_a((i - j) mod n_a), c_a(t) = exp(-2 beta R_a^2 (1 - cos(2 pi t / n_a))).
Each circulant is diagonalised by the discrete Fourier modes, with real
eigenvalues lambda_a(m) = sum_t c_a(t) cos(2 pi t m / n_a).

Consequences used by the tests:
* every eigenvalue of K is a product prod_a lambda_a(m_a);
* q = K 1 is the constant prod_a lambda_a(0), so for every alpha the
  normalisation of Sec. 2.1 gives s = q^-1/2 and M = K / q;
* K V is computed exactly at any grid size by multiplying along each axis.

Point order: grid indices in C order, the first axis varying slowest.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np


def circulant_first_row(n: int, R: float, beta: float) -> np.ndarray:
    t = np.arange(n)
    return np.exp(-2.0 * float(beta) * float(R) ** 2 * (1.0 - np.cos(2.0 * np.pi * t / n)))


def circulant_eigs(n: int, R: float, beta: float) -> np.ndarray:
    """lambda(m) = sum_t c(t) cos(2 pi t m / n), m = 0 .. n-1."""
    c = circulant_first_row(n, R, beta)
    t = np.arange(n)
    m = np.arange(n)
    return np.cos(2.0 * np.pi * np.outer(m, t) / n) @ c


def _radii(counts: Sequence[int], radii) -> np.ndarray:
    return np.ones(len(counts)) if radii is None else np.asarray(radii, dtype=np.float64)


def kernel_eigs(counts: Sequence[int], beta: float, radii=None) -> np.ndarray:
    """All eigenvalues of K on the grid (unsorted, Kronecker order)."""
    R = _radii(counts, radii)
    ev = np.ones(1)
    for n, r in zip(counts, R):
        ev = np.multiply.outer(ev, circulant_eigs(int(n), r, beta)).reshape(-1)
    return ev


def degree(counts: Sequence[int], beta: float, radii=None) -> float:
    """The constant row sum q = prod_a lambda_a(0)."""
    R = _radii(counts, radii)
    return float(np.prod([circulant_eigs(int(n), r, beta)[0] for n, r in zip(counts, R)]))


def operator_eigs(counts: Sequence[int], beta: float, radii=None) -> np.ndarray:
    """Eigenvalues of M = K / q, sorted descending."""
    ev = kernel_eigs(counts, beta, radii) / degree(counts, beta, radii)
    return np.sort(ev)[::-1]


def kernel_apply(counts: Sequence[int], beta: float, V: np.ndarray, radii=None) -> np.ndarray:
    """K V for the grid points, exactly, by one circulant product per axis."""
    R = _radii(counts, radii)
    counts = [int(n) for n in counts]
    V = np.asarray(V, dtype=np.float64)
    squeeze = V.ndim == 1
    if squeeze:
        V = V[:, None]
    b = V.shape[1]
    T = V.reshape(*counts, b)
    for a, (n, r) in enumerate(zip(counts, R)):
        c = circulant_first_row(n, r, beta)
        idx = (np.arange(n)[:, None] - np.arange(n)[None, :]) % n
        C = c[idx]
        T = np.moveaxis(np.tensordot(C, T, axes=([1], [a])), 0, a)
    out = T.reshape(-1, b)
    return out[:, 0] if squeeze else out


def fourier_mode(counts: Sequence[int], modes: Sequence[int], kind: str = "cos") -> np.ndarray:
    """Real Fourier mode prod_a e^{i 2 pi m_a i_a / n_a}: its real or imaginary part.

    Each such vector is an exact eigenvector of K on the grid.
    """
    axes = [2.0 * np.pi * m * np.arange(n) / n for n, m in zip(counts, modes)]
    mesh = np.meshgrid(*axes, indexing="ij")
    phase = sum(mesh)
    v = np.cos(phase) if kind == "cos" else np.sin(phase)
    return v.reshape(-1)
