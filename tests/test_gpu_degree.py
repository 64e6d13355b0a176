"""Parity of fd_degree (normalisation passes) with the oracle.

q = K 1, d = q^-alpha (K q^-alpha), s = q^-alpha d^-1/2 and S_off = sum(q) - N
(Sec. 2.1, Sec. 2.3) against the float64 oracle, relative 2-norm error
<= 1e-5 per vector.  Full size: the Markov operator built from the GPU's
own w and d is row-stochastic (P 1 = 1), and on a grid torus q is the
closed-form constant.
"""
import numpy as np
import pytest
import torch

from gpu_util import TOL_F32, case, device, rel_fro, to_dev, to_np
from oracle import normalise as on
from oracle import torus_grid as tg
from paper_2609_38198_amd import _lib as fd
from paper_2609_38198_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("alpha", [0.0, 0.5, 1.0])
def test_torus2_normalisation(alpha):
    w = inputs.torus2()
    dev = device()
    case(f"degree torus2 alpha={alpha}")
    deg = fd.fd_degree(to_dev(w.X, dev), 8.0, alpha)
    ref = on.normalise(w.X, 8.0, alpha)
    assert rel_fro(to_np(deg.q), ref.q) <= TOL_F32
    assert rel_fro(to_np(deg.d), ref.d) <= TOL_F32
    assert rel_fro(to_np(deg.s), ref.s) <= TOL_F32
    s_off = float(to_np(deg.s_off)[0])
    assert abs(s_off - ref.s_off) <= TOL_F32 * float(ref.q.sum())


@pytest.mark.parametrize("beta", [0.5, 8.0])
def test_ragged_sizes(beta):
    rng = np.random.default_rng(7)
    X = rng.normal(size=(1001, 6)).astype(np.float32)
    X -= X.mean(0)
    dev = device()
    case(f"degree ragged N=1001 beta={beta}")
    deg = fd.fd_degree(to_dev(X, dev), beta, 0.5)
    ref = on.normalise(X, beta, 0.5)
    for name in ("q", "d", "s"):
        assert rel_fro(to_np(getattr(deg, name)), getattr(ref, name)) <= TOL_F32


@pytest.mark.parametrize("beta", [0.5, 2.0, 8.0])
def test_torus6_full_size_markov_rows_sum_to_one(beta):
    w = inputs.torus6()
    dev = device()
    X = to_dev(w.X, dev)
    case(f"degree torus6 N=65536 beta={beta}")
    deg = fd.fd_degree(X, beta, 0.5)
    q = deg.q
    wv = q.double().pow(-0.5).float()
    # P 1 = diag(d)^-1 diag(w) K diag(w) 1
    sl = (wv.double() / deg.d.double()).float()
    ones = torch.ones((w.N, 1), dtype=torch.float32, device=dev)
    P1 = to_np(fd.fd_kernel_matmul(X, None, beta, ones, sl=sl, sr=wv))[:, 0]
    assert np.abs(P1 - 1.0).max() <= 1e-5
    # sampled rows of q against the oracle
    rows = np.random.default_rng(3).choice(w.N, 256, replace=False)
    from oracle import kernel as ok
    qref = ok.kernel_matmul(w.X, None, beta, np.ones(w.N), rows=rows, threads=8)
    assert rel_fro(to_np(q)[rows], qref) <= TOL_F32


@pytest.mark.parametrize("D", [1, 5, 9, 14, 27, 31, 33, 63])
def test_every_feature_width(D):
    rng = np.random.default_rng(2000 + D)
    X = (rng.normal(size=(900, D)) * 0.5).astype(np.float32)
    X -= X.mean(0)
    dev = device()
    case(f"degree feature width D={D}")
    deg = fd.fd_degree(to_dev(X, dev), 2.0 / D, 0.5)
    ref = on.normalise(X, 2.0 / D, 0.5)
    for name in ("q", "d", "s"):
        assert rel_fro(to_np(getattr(deg, name)), getattr(ref, name)) <= TOL_F32


def test_grid_torus_constant_degree():
    counts = (8, 8, 8, 8, 4, 4)
    X = inputs.grid_torus_points(counts).astype(np.float32)
    dev = device()
    case("degree grid torus 65536")
    deg = fd.fd_degree(to_dev(X, dev), 1.0, 0.5)
    q0 = tg.degree(counts, 1.0)
    q = to_np(deg.q)
    assert np.abs(q / q0 - 1).max() <= 1e-5
    s = to_np(deg.s)
    assert np.abs(s * np.sqrt(q0) - 1).max() <= 1e-5


def test_bf16_normalisation():
    # bfloat16 X: exact bfloat16 products in the distance contraction, float32
    # sums, so the normalisation meets the float32 tolerance
    s = inputs.stress(N=4096)
    dev = device()
    beta = s.betas[0]
    case("degree bf16 N=4096 D=64")
    deg = fd.fd_degree(to_dev(s.X, dev), beta, 0.5)
    ref = on.normalise(s.X_f64(), beta, 0.5)
    for name in ("q", "d", "s"):
        assert rel_fro(to_np(getattr(deg, name)), getattr(ref, name)) <= TOL_F32


# Block counts of the symmetric row sums (blocks of 512 points): one block,
# even and odd counts (the pairing of blocks differs), ragged last blocks.
@pytest.mark.parametrize("N", [1, 2, 17, 511, 513, 1536, 2560, 3072, 3583])
def test_symmetric_block_counts(N):
    rng = np.random.default_rng(31 + N)
    X = rng.normal(size=(N, 7)).astype(np.float32)
    X -= X.mean(0)
    dev = device()
    case(f"degree symmetric row sums N={N}")
    for beta in (0.05, 1.0):
        deg = fd.fd_degree(to_dev(X, dev), beta, 0.5)
        ref = on.normalise(X, beta, 0.5)
        for name in ("q", "d", "s"):
            assert rel_fro(to_np(getattr(deg, name)), getattr(ref, name)) <= TOL_F32, (beta, name)


def test_symmetric_row_sums_match_plain_product_and_repeat_bitwise():
    # q from the symmetric row sums against K 1 from the fused product (a
    # separate kernel that evaluates every entry), and two calls bit for bit
    w = inputs.torus6()
    dev = device()
    X = to_dev(w.X, dev)
    case("degree symmetric vs product K 1, torus6 N=65536")
    ones = torch.ones((w.N, 1), dtype=torch.float32, device=dev)
    for beta in (0.5, 8.0):
        a = fd.fd_degree(X, beta, 0.5)
        b = fd.fd_degree(X, beta, 0.5)
        torch.cuda.synchronize()
        for name in ("q", "d", "s"):
            assert torch.equal(getattr(a, name), getattr(b, name)), name
        k1 = to_np(fd.fd_kernel_matmul(X, None, beta, ones))[:, 0]
        q = to_np(a.q)
        # both evaluate the exponent in float32 in the Gram form, with a rounding
        # of about 2^-24 * 2 beta log2(e) max ||x||^2 (in log2 units) that
        # depends on the evaluation order: entries may differ by twice that
        bound = 2 * 2.0**-24 * 2 * beta * np.log2(np.e) * float((w.X.astype(np.float64) ** 2).sum(1).max())
        assert rel_fro(q, k1) <= 1e-6
        assert np.abs(q / k1 - 1.0).max() <= bound * np.log(2) + 1e-6
