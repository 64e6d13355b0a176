"""Seeded synthetic inputs for the diffusion-map kernel workloads.

This module is shared by the tests, the benchmark and the smoke check.  It
draws point clouds and right-hand-side blocks and nothing else: no kernel
value, normalisation, product or eigenvalue is computed here.  Both the
HIP path and the CPU oracle receive the arrays it returns.

All randomness comes from ``numpy.random.default_rng(seed)`` (PCG64).

Workloads (each is a reading of the workload description; the readings are
recorded in the design notes):

* ``torus2``   flat 2-torus, N=2048, angles ~ U[0, 2pi), embedded in R^4 as
               (cos t1, sin t1, cos t2, sin t2); beta=8, b=8, k=16.
* ``torus6``   flat 6-torus, N=65536, six angles embedded in R^12;
               b=16, beta in {0.5, 1, 2, 4, 8}.
* ``torus6n``  ``torus6`` with N=262144 plus N(0, 0.01^2) noise per
               coordinate; b=32, k=64; continuation over nested prefixes.
* ``molecule`` N=1048576; two angles from a 4-component von Mises mixture
               (kappa=4) mapped through a fixed seeded 2-layer tanh MLP
               (4 -> 64 -> 30) plus N(0, 0.05^2) noise; b=32, k=64.
* ``stress``   N=2097152 standard Gaussian in R^64 projected onto a seeded
               8-dim subspace plus N(0, 0.1^2) noise, stored as bfloat16;
               b=64, beta = 1/median squared distance of a 4096-point
               subsample.
* ``grid_torus`` points on a regular grid of a flat torus with given radii
               (companion inputs with a closed-form spectrum).
* ``torus6_paper`` the paper's own T^6 set-up (Sec. 3): radii
               (1.00, 1.08, 1.17, 1.27, 1.38, 1.50), angles from seed 42,
               zero-padded to D=32; beta=1 for the raw kernel application
               of App. B (b in {1, 8}); the angles are kept for the
               recovery score of the leading doublet.

Every point cloud is centred in float64 (the method expects centred
observations, Sec. 2.1 and the T^6 experiment) and then cast.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

TWO_PI = 2.0 * math.pi


@dataclasses.dataclass
class Workload:
    """One synthetic workload: the points and the solver parameters."""

    name: str
    X: np.ndarray            # (N, D) float32, or uint16 holding bfloat16 bits
    dtype: str               # "f32" or "bf16"
    betas: tuple             # bandwidths to run
    b: int                   # block width
    k: Optional[int]         # eigenpairs requested (None: product only)
    alpha: float = 0.5
    extra: dict = dataclasses.field(default_factory=dict)

    @property
    def N(self) -> int:
        return int(self.X.shape[0])

    @property
    def D(self) -> int:
        return int(self.X.shape[1])

    def X_f64(self) -> np.ndarray:
        """The exact values the kernel sees, widened to float64."""
        if self.dtype == "bf16":
            return bf16_bits_to_f64(self.X)
        return self.X.astype(np.float64)


# --------------------------------------------------------------------------
# element helpers (storage conversions only)
# --------------------------------------------------------------------------

def centre_f64(X: np.ndarray) -> np.ndarray:
    X = np.asarray(X, dtype=np.float64)
    return X - X.mean(axis=0, keepdims=True)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returns the 16-bit patterns as uint16.  NaN/Inf do not occur in the
    generated data and are not special-cased beyond keeping NaN a NaN.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = (u + 0x7FFF + lsb) >> 16
    out = rounded.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(bits).astype(np.float64)


def median_sq_distance(X: np.ndarray, n_sub: int = 4096, seed: int = 0) -> float:
    """Median squared distance over distinct pairs of a seeded subsample.

    This is the bandwidth recipe of the ``stress`` workload (beta is its
    reciprocal); it only sets an input parameter.
    """
    X = np.asarray(X, dtype=np.float64)
    rng = np.random.default_rng(seed)
    idx = rng.choice(X.shape[0], size=min(n_sub, X.shape[0]), replace=False)
    S = X[np.sort(idx)]
    vals = []
    for i in range(S.shape[0] - 1):
        diff = S[i + 1:] - S[i]
        vals.append(np.einsum("ij,ij->i", diff, diff))
    return float(np.median(np.concatenate(vals)))


# --------------------------------------------------------------------------
# point clouds
# --------------------------------------------------------------------------

def torus_points(N: int, n_angles: int, seed: int = 0, radii: Optional[Sequence[float]] = None,
                 noise: float = 0.0, pad_to: Optional[int] = None) -> np.ndarray:
    """Uniform samples of a flat n-torus embedded as (R cos t, R sin t) pairs.

    Column order is (cos t1, sin t1, cos t2, sin t2, ...).  Angles are drawn
    first as one (N, n_angles) block, noise afterwards from the same
    generator.  Returns centred float64.
    """
    rng = np.random.default_rng(seed)
    theta = rng.uniform(0.0, TWO_PI, size=(N, n_angles))
    R = np.ones(n_angles) if radii is None else np.asarray(radii, dtype=np.float64)
    X = np.empty((N, 2 * n_angles), dtype=np.float64)
    X[:, 0::2] = R * np.cos(theta)
    X[:, 1::2] = R * np.sin(theta)
    if noise > 0.0:
        X += rng.normal(0.0, noise, size=X.shape)
    if pad_to is not None and pad_to > X.shape[1]:
        X = np.concatenate([X, np.zeros((N, pad_to - X.shape[1]))], axis=1)
    return centre_f64(X)


def grid_torus_points(counts: Sequence[int], radii: Optional[Sequence[float]] = None) -> np.ndarray:
    """Regular grid on a flat torus: angle a takes values 2 pi i / counts[a].

    Points are ordered with the first angle varying slowest (C order over
    the grid indices).  Returns float64 (the grid is centred by symmetry;
    it is centred again numerically).
    """
    counts = [int(c) for c in counts]
    R = np.ones(len(counts)) if radii is None else np.asarray(radii, dtype=np.float64)
    axes = [TWO_PI * np.arange(c) / c for c in counts]
    mesh = np.meshgrid(*axes, indexing="ij")
    theta = np.stack([m.reshape(-1) for m in mesh], axis=1)
    X = np.empty((theta.shape[0], 2 * len(counts)), dtype=np.float64)
    X[:, 0::2] = R * np.cos(theta)
    X[:, 1::2] = R * np.sin(theta)
    return centre_f64(X)


def molecule_points(N: int, seed: int = 0) -> np.ndarray:
    """Two von Mises mixture angles -> (cos, sin) features -> tanh MLP -> noise.

    Reading: 4 components with means on a 2x2 grid of spacing pi shifted by
    a seeded U[0, 2 pi)^2 offset, independent von Mises(kappa=4) on each
    angle, equal weights; MLP h = tanh(f W1), y = h W2 without biases,
    W1 ~ N(0, 1/4), W2 ~ N(0, 1/64); then N(0, 0.05^2) noise in R^30.
    """
    rng = np.random.default_rng(seed)
    offset = rng.uniform(0.0, TWO_PI, size=2)
    means = np.array([[offset[0] + math.pi * a, offset[1] + math.pi * c]
                      for a in (0, 1) for c in (0, 1)]) % TWO_PI
    W1 = rng.normal(0.0, math.sqrt(1.0 / 4.0), size=(4, 64))
    W2 = rng.normal(0.0, math.sqrt(1.0 / 64.0), size=(64, 30))
    comp = rng.integers(0, 4, size=N)
    phi = rng.vonmises(means[comp, 0], 4.0)
    psi = rng.vonmises(means[comp, 1], 4.0)
    f = np.stack([np.cos(phi), np.sin(phi), np.cos(psi), np.sin(psi)], axis=1)
    Y = np.tanh(f @ W1) @ W2
    Y += rng.normal(0.0, 0.05, size=Y.shape)
    return centre_f64(Y)


def stress_points(N: int, seed: int = 0, D: int = 64, sub_dim: int = 8,
                  noise: float = 0.1) -> np.ndarray:
    """Gaussian in R^D projected on a seeded sub_dim subspace, plus noise.

    X = G U U^T + noise * E with U the Q factor of a seeded D x sub_dim
    Gaussian.  Generated in row chunks to bound memory.  Returns float64.
    """
    rng = np.random.default_rng(seed)
    U, _ = np.linalg.qr(rng.normal(size=(D, sub_dim)))
    P = U @ U.T
    X = np.empty((N, D), dtype=np.float64)
    chunk = 1 << 18
    for s in range(0, N, chunk):
        e = min(N, s + chunk)
        G = rng.standard_normal((e - s, D))
        E = rng.standard_normal((e - s, D))
        X[s:e] = G @ P + noise * E
    return centre_f64(X)


def random_block(N: int, b: int, seed: int = 1) -> np.ndarray:
    """Right-hand-side block V ~ N(0, 1), float32, row-major N x b."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((N, b)).astype(np.float32)


# --------------------------------------------------------------------------
# named workloads
# --------------------------------------------------------------------------

def torus2(N: int = 2048, seed: int = 0) -> Workload:
    X = torus_points(N, 2, seed=seed).astype(np.float32)
    return Workload("torus2", X, "f32", (8.0,), 8, 16)


def torus6(N: int = 65536, seed: int = 0) -> Workload:
    X = torus_points(N, 6, seed=seed).astype(np.float32)
    return Workload("torus6", X, "f32", (0.5, 1.0, 2.0, 4.0, 8.0), 16, None)


T6_RADII = (1.00, 1.08, 1.17, 1.27, 1.38, 1.50)


def torus6_paper(N: int = 65536, seed: int = 42) -> Workload:
    # the angles are drawn exactly as torus_points draws them (same seed,
    # same first call), and kept
    theta = np.random.default_rng(seed).uniform(0.0, TWO_PI, size=(N, 6))
    X = torus_points(N, 6, seed=seed, radii=T6_RADII, pad_to=32).astype(np.float32)
    return Workload("torus6_paper", X, "f32", (1.0,), 8, 3, extra={"theta": theta})


def torus6_noisy(N: int = 262144, seed: int = 0) -> Workload:
    X = torus_points(N, 6, seed=seed, noise=0.01).astype(np.float32)
    return Workload("torus6n", X, "f32", (0.5, 1.0, 2.0, 4.0, 8.0), 32, 64,
                    extra={"n_ladder": (16384, 65536, 262144)})


def molecule(N: int = 1 << 20, seed: int = 0) -> Workload:
    Xd = molecule_points(N, seed=seed)
    X = Xd.astype(np.float32)
    beta = 1.0 / median_sq_distance(X, 4096, seed)
    return Workload("molecule", X, "f32", (beta,), 32, 64)


def stress(N: int = 1 << 21, seed: int = 0) -> Workload:
    Xd = stress_points(N, seed=seed)
    bits = f32_to_bf16_bits(Xd.astype(np.float32))
    del Xd
    beta = 1.0 / median_sq_distance(bf16_bits_to_f64(bits), 4096, seed)
    return Workload("stress", bits, "bf16", (beta,), 64, 64, extra={"iters": 20})


WORKLOADS = {
    "torus2": torus2,
    "torus6": torus6,
    "torus6n": torus6_noisy,
    "molecule": molecule,
    "stress": stress,
    "torus6_paper": torus6_paper,
}
