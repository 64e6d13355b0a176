"""Gaussian affinity and its scaled products, float64 (test infrastructure).

Sec. 2.1, eq. kernel: K = exp(-beta H), H the matrix of pairwise squared
Euclidean distances.  H is written in the difference form
H_ij = sum_k (x_ik - x_jk)^2, straight from its definition (not the Gram
form of eq. rbf_gram that the fast path evaluates).

Sec. 2.1 eq. matmat and Sec. 2.2 eq. tiled_rbf: the operator applied to a
block is Y = diag(sl) K diag(sr) V.  Rows of Y are independent, so the
product may be evaluated for any subset of rows; that is how it is checked
at sizes where the full N x N matrix does not fit in memory.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Sequence

import numpy as np


def sq_distances(Xr: np.ndarray, Xc: np.ndarray) -> np.ndarray:
    """H_ij = sum_k (Xr[i,k] - Xc[j,k])^2 in float64 (difference form)."""
    Xr = np.asarray(Xr, dtype=np.float64)
    Xc = np.asarray(Xc, dtype=np.float64)
    H = np.zeros((Xr.shape[0], Xc.shape[0]), dtype=np.float64)
    for k in range(Xr.shape[1]):
        diff = Xr[:, k, None] - Xc[None, :, k]
        H += diff * diff
    return H


def gaussian_kernel(Xr: np.ndarray, Xc: Optional[np.ndarray], beta: float) -> np.ndarray:
    """K_ij = exp(-beta * ||xr_i - xc_j||^2)   (Sec. 2.1, eq. kernel)."""
    if Xc is None:
        Xc = Xr
    return np.exp(-float(beta) * sq_distances(Xr, Xc))


def kernel_matmul(Xr: np.ndarray, Xc: Optional[np.ndarray], beta: float, V: np.ndarray,
                  sl: Optional[np.ndarray] = None, sr: Optional[np.ndarray] = None,
                  rows: Optional[Sequence[int]] = None, block: int = 256,
                  threads: int = 1) -> np.ndarray:
    """Y = diag(sl) K(Xr, Xc) diag(sr) V, restricted to ``rows`` if given.

    Sec. 2.1 eq. matmat (scaled block product) and Sec. 2.2 eq. tiled_rbf
    (the rectangular application K(X_I, X_J) V_J).  sl / sr default to ones.
    ``rows`` selects output rows of Xr (the other rows are not computed).
    Row blocks are independent evaluations of the same definition; with
    ``threads`` > 1 they run on a thread pool (numpy releases the GIL).
    Returns float64 of shape (len(rows) or Nr, b).
    """
    Xr = np.asarray(Xr, dtype=np.float64)
    Xc = Xr if Xc is None else np.asarray(Xc, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    squeeze = V.ndim == 1
    if squeeze:
        V = V[:, None]
    if V.shape[0] != Xc.shape[0]:
        raise ValueError("V must have one row per column point")
    W = V if sr is None else np.asarray(sr, dtype=np.float64)[:, None] * V
    idx = np.arange(Xr.shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    slv = None if sl is None else np.asarray(sl, dtype=np.float64)
    Y = np.empty((idx.shape[0], V.shape[1]), dtype=np.float64)

    def one(start: int) -> None:
        sel = idx[start:start + block]
        K = gaussian_kernel(Xr[sel], Xc, beta)
        out = K @ W
        if slv is not None:
            out *= slv[sel, None]
        Y[start:start + block] = out

    starts = range(0, idx.shape[0], block)
    if threads > 1:
        with ThreadPoolExecutor(max_workers=threads) as pool:
            list(pool.map(one, starts))
    else:
        for s in starts:
            one(s)
    return Y[:, 0] if squeeze else Y
