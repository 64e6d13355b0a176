"""Coifman-Lafon normalisation, float64 (test infrastructure).

Sec. 2.1: q = K 1; K_alpha = diag(q)^-alpha K diag(q)^-alpha; the degree
d = K_alpha 1; P = diag(d)^-1 K_alpha is row-stochastic; it is similar to the
symmetric M = diag(d)^1/2 P diag(d)^-1/2 = diag(s) K diag(s) with
s = q^-alpha * d^-1/2 (eq. symmetric).

The definition of d is written twice in the paper; the second statement
drops the trailing "times the ones vector".  The reading taken here is
d = K_alpha 1 as in the first statement.

S_off = sum_{i != j} K_ij (Sec. 2.3, before eq. neff) equals sum(q) - N
because K_ii = 1.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

from .kernel import gaussian_kernel, kernel_matmul


@dataclass
class Normalisation:
    q: np.ndarray      # K 1
    w: np.ndarray      # q^-alpha
    d: np.ndarray      # K_alpha 1 = w * (K w)
    s: np.ndarray      # w * d^-1/2
    s_off: float       # sum_{i != j} K_ij


def normalise(X: np.ndarray, beta: float, alpha: float, rows_block: int = 256,
              threads: int = 1) -> Normalisation:
    """q, q^-alpha, d and s from their definitions (Sec. 2.1).

    Uses two kernel applications (V = 1, then V = q^-alpha), never the dense
    N x N matrix, so it runs at the workloads' full sizes.
    """
    X = np.asarray(X, dtype=np.float64)
    N = X.shape[0]
    ones = np.ones(N)
    q = kernel_matmul(X, None, beta, ones, block=rows_block, threads=threads)
    w = q ** (-float(alpha))
    t = kernel_matmul(X, None, beta, w, block=rows_block, threads=threads)
    d = w * t
    s = w / np.sqrt(d)
    s_off = float(np.sum(q) - N)
    return Normalisation(q=q, w=w, d=d, s=s, s_off=s_off)


def off_diagonal_mass(K: np.ndarray) -> float:
    """S_off = sum over i != j of K_ij, from a dense K (Sec. 2.3)."""
    return float(K.sum() - np.trace(K))


def operator_M(X: np.ndarray, beta: float, alpha: float,
               K: Optional[np.ndarray] = None) -> tuple[np.ndarray, Normalisation]:
    """Dense symmetric diffusion operator M = diag(s) K diag(s) (eq. symmetric)."""
    X = np.asarray(X, dtype=np.float64)
    if K is None:
        K = gaussian_kernel(X, None, beta)
    q = K.sum(axis=1)
    w = q ** (-float(alpha))
    d = w * (K @ w)
    s = w / np.sqrt(d)
    M = s[:, None] * K * s[None, :]
    nrm = Normalisation(q=q, w=w, d=d, s=s, s_off=off_diagonal_mass(K))
    return M, nrm


def operator_P(X: np.ndarray, beta: float, alpha: float,
               K: Optional[np.ndarray] = None) -> np.ndarray:
    """Dense row-stochastic Markov operator P = diag(d)^-1 K_alpha (Sec. 2.1)."""
    X = np.asarray(X, dtype=np.float64)
    if K is None:
        K = gaussian_kernel(X, None, beta)
    q = K.sum(axis=1)
    w = q ** (-float(alpha))
    Ka = w[:, None] * K * w[None, :]
    d = Ka.sum(axis=1)
    return Ka / d[:, None]
