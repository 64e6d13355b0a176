"""Spectral diagnostics, float64 (test infrastructure).

* Perron gap g_P = (lambda_0 - lambda_1) / |lambda_0| and the precision wall
  g_P > kappa_P * eta with kappa_P = 10 (Sec. 2.3, eqs. vmach, perronwall);
  eta per data type from the footnote to eq. perronwall.
* Smooth barrier V_mach = (kappa_P eta / g_P)^p with p = 6 (eq. vmach).
* Principal angles between subspaces (LAPACK-based, through scipy).
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
