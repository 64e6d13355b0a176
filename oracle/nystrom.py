"""Nystrom extension of Markov eigenvectors, float64 (test infrastructure).

Sec. 1 and Sec. 2.3 extend an eigenspace from a subsample to a larger
sample with the Nystrom extension but give no formula.  The one used here
follows from the definitions of Sec. 2.1: with w = q^-alpha over the old
sample, row i of P psi = lambda psi reads

    psi_i = (1/lambda) * sum_j K_ij w_j psi_j / sum_j K_ij w_j,

(the factor q_i^-alpha cancels).  Evaluating the right-hand side at a new
point x gives psi(x).  On the old points it returns psi itself.
"""
from __future__ import annotations

import numpy as np

from .kernel import kernel_matmul


def nystrom_extend(X_old: np.ndarray, X_new: np.ndarray, beta: float, alpha: float,
                   psi: np.ndarray, evals: np.ndarray, q_old: np.ndarray | None = None,
                   threads: int = 1) -> np.ndarray:
    """Extend Markov eigenvectors psi (n_old x k) to the points X_new."""
    X_old = np.asarray(X_old, dtype=np.float64)
    X_new = np.asarray(X_new, dtype=np.float64)
    psi = np.asarray(psi, dtype=np.float64)
    if psi.ndim == 1:
        psi = psi[:, None]
    evals = np.atleast_1d(np.asarray(evals, dtype=np.float64))
    if q_old is None:
        q_old = kernel_matmul(X_old, None, beta, np.ones(X_old.shape[0]), threads=threads)
    w = np.asarray(q_old, dtype=np.float64) ** (-float(alpha))
    V = np.concatenate([w[:, None], w[:, None] * psi], axis=1)
    T = kernel_matmul(X_new, X_old, beta, V, threads=threads)
    return T[:, 1:] / T[:, :1] / evals[None, :]
