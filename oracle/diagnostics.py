"""Spectral diagnostics, float64 (test infrastructure).

* Perron gap g_P = (lambda_0 - lambda_1) / |lambda_0| and the precision wall
  g_P > kappa_P * eta with kappa_P = 10 (Sec. 2.3, eqs. vmach, perronwall);
  eta per data type from the footnote to eq. perronwall.
* Smooth barrier V_mach = (kappa_P eta / g_P)^p with p = 6 (eq. vmach).
* Principal angles between subspaces (LAPACK-based, through scipy).
* Rotation-invariant subspace overlap of Sec. 3 (the T^6 recovery score, in
  the footnote to the discussion of its figure c): with A and B the column
  blocks of two subspaces and G_AA, G_BB, G_AB their centred covariance
  blocks, C = G_AA^-1/2 G_AB G_BB^-1/2 and the score is sum_ij C_ij^2 / 2 for
  two-dimensional blocks (the squared RV coefficient).  Reading: for blocks
  of other widths the sum is divided by the smaller width, so that the score
  is 1 when one span contains the other and 0 when they are orthogonal.
"""
from __future__ import annotations

import numpy as np
import scipy.linalg

ETA = {"bf16": 8e-3, "tf32": 1e-3, "fp32": 1e-7, "fp64": 2.22e-16}
KAPPA_P = 10.0
P_EXPONENT = 6


def perron_gap(evals: np.ndarray) -> float:
    ev = np.asarray(evals, dtype=np.float64)
    return float((ev[0] - ev[1]) / abs(ev[0]))


def wall_admissible(gap: float, dtype: str = "fp32") -> bool:
    """Hard admissibility g_P > kappa_P * eta (eq. perronwall)."""
    return bool(gap > KAPPA_P * ETA[dtype])


def v_mach(gap: float, dtype: str = "fp32") -> float:
    return float((KAPPA_P * ETA[dtype] / gap) ** P_EXPONENT)


def principal_angles(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Principal angles (radians, descending) between span(A) and span(B)."""
    return scipy.linalg.subspace_angles(np.asarray(A, dtype=np.float64),
                                        np.asarray(B, dtype=np.float64))


def _inv_sqrt_spd(G: np.ndarray) -> np.ndarray:
    w, U = np.linalg.eigh(G)
    return (U / np.sqrt(w)) @ U.T


def rv_overlap(A: np.ndarray, B: np.ndarray) -> float:
    """Whitened cross-covariance overlap of span(A) and span(B) in [0, 1]."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    if A.ndim == 1:
        A = A[:, None]
    if B.ndim == 1:
        B = B[:, None]
    A = A - A.mean(axis=0)
    B = B - B.mean(axis=0)
    C = _inv_sqrt_spd(A.T @ A) @ (A.T @ B) @ _inv_sqrt_spd(B.T @ B)
    return float((C ** 2).sum() / min(A.shape[1], B.shape[1]))
