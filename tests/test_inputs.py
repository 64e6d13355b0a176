"""Seeded input generators: reproducible, centred, right shapes (CPU only)."""
import numpy as np
import pytest
import torch

from paper_2609_38198_amd import inputs


def test_torus2_shape_seed_centring():
    a = inputs.torus2()
    b = inputs.torus2()
    assert a.X.shape == (2048, 4) and a.X.dtype == np.float32
    np.testing.assert_array_equal(a.X, b.X)
    assert np.abs(a.X.astype(np.float64).mean(0)).max() < 1e-7
    assert a.betas == (8.0,) and a.b == 8 and a.k == 16
    # recipe: angles from default_rng(0) as one (N, 2) block, (cos, sin) pairs, centred
    th = np.random.default_rng(0).uniform(0, 2 * np.pi, (2048, 2))
    raw = np.stack([np.cos(th[:, 0]), np.sin(th[:, 0]), np.cos(th[:, 1]), np.sin(th[:, 1])], 1)
    np.testing.assert_allclose(inputs.torus_points(2048, 2, seed=0), raw - raw.mean(0), atol=1e-15)


def test_torus6_and_noisy_prefix_structure():
    w = inputs.torus6(N=4096)
    assert w.X.shape == (4096, 12) and w.b == 16 and w.k is None
    n = inputs.torus6_noisy(N=4096)
    assert n.X.shape == (4096, 12) and n.b == 32 and n.k == 64
    # noise is small relative to the manifold
    assert 0.0 < np.abs(n.X - w.X).max() < 0.1


def test_molecule_small():
    m = inputs.molecule(N=8192)
    assert m.X.shape == (8192, 30) and np.isfinite(m.X).all()
    assert 0 < m.betas[0] < 10


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).normal(size=10000).astype(np.float32) * 3
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0, 65504.0]   # ties and edge values
    bits = inputs.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bits, ref)
    back = inputs.bf16_bits_to_f32(bits)
    np.testing.assert_array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_stress_small_is_bf16():
    s = inputs.stress(N=8192)
    assert s.X.dtype == np.uint16 and s.X.shape == (8192, 64) and s.dtype == "bf16"
    Xd = s.X_f64()
    assert np.isfinite(Xd).all()
    assert s.betas[0] > 0


def test_grid_torus_points_order():
    X = inputs.grid_torus_points((4, 3))
    assert X.shape == (12, 4)
    # second axis varies fastest
    assert np.allclose(X[0, :2], X[1, :2]) and not np.allclose(X[0, 2:], X[1, 2:])


def test_median_sq_distance_small():
    X = np.array([[0.0], [1.0], [3.0]])
    # pairwise squared distances 1, 9, 4 -> median 4
    assert inputs.median_sq_distance(X, n_sub=3) == pytest.approx(4.0)


def test_torus6_paper_layout():
    # Sec. 3: radii (1.00 ... 1.50) in R^12, zero-padded to D=32, centred,
    # angles kept for the recovery score
    w = inputs.torus6_paper(2000)
    assert w.X.shape == (2000, 32) and w.X.dtype == np.float32
    assert np.all(w.X[:, 12:] == 0.0)
    X = w.X.astype(np.float64)
    np.testing.assert_allclose(X.mean(0), 0.0, atol=1e-6)
    th = w.extra["theta"]
    for a, R in enumerate(inputs.T6_RADII):
        raw = np.stack([R * np.cos(th[:, a]), R * np.sin(th[:, a])], 1)
        np.testing.assert_allclose(X[:, 2 * a:2 * a + 2], raw - raw.mean(0), atol=1e-6)
