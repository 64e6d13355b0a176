"""Dense eigensolve of the symmetric diffusion operator, float64.

Test infrastructure.  Sec. 2.1 (eq. symmetric): P and M share eigenvalues, so
the spectrum is taken from the symmetric M with LAPACK (numpy ``eigh``,
divide and conquer).  Sec. 2.3: a probe returns the Perron mode with the
requested nontrivial modes; the Markov right eigenvectors follow by the
diagonal rescale psi = d^-1/2 phi (last paragraph of Sec. 2.3, and
M = diag(d)^1/2 P diag(d)^-1/2).

Reading: ``k`` counts every returned pair including the Perron pair.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .normalise import Normalisation, operator_M


@dataclass
class Spectrum:
    evals: np.ndarray   # (k,) descending
    phi: np.ndarray     # (N, k) orthonormal eigenvectors of M
    psi: np.ndarray     # (N, k) Markov right eigenvectors d^-1/2 phi
    norm: Normalisation


def top_eigenpairs(M: np.ndarray, k: int) -> tuple[np.ndarray, np.ndarray]:
    """Largest k eigenvalues (descending) and eigenvectors of symmetric M."""
    w, V = np.linalg.eigh(M)
    order = np.argsort(w)[::-1][:k]
    return w[order], V[:, order]


def markov_eigvecs(phi: np.ndarray, d: np.ndarray) -> np.ndarray:
    """psi = diag(d)^-1/2 phi."""
    return phi / np.sqrt(d)[:, None]


def sign_fix(V: np.ndarray) -> np.ndarray:
    """Flip each column so its largest-magnitude entry is positive (reporting)."""
    V = np.array(V, dtype=np.float64, copy=True)
    idx = np.argmax(np.abs(V), axis=0)
    sgn = np.sign(V[idx, np.arange(V.shape[1])])
    sgn[sgn == 0] = 1.0
    return V * sgn


def spectrum(X: np.ndarray, beta: float, alpha: float, k: int) -> Spectrum:
    """Top-k eigenpairs of M for the points X (dense; small N only)."""
    M, nrm = operator_M(X, beta, alpha)
    evals, phi = top_eigenpairs(M, k)
    return Spectrum(evals=evals, phi=phi, psi=markov_eigvecs(phi, nrm.d), norm=nrm)
