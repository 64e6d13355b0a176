"""Error paths on the GPU: non-finite inputs, the float32 exponent range and
rank-deficient warm starts.

A NaN or infinite coordinate makes every output of the asynchronous entry
points NaN (fd_kernel_matmul, fd_degree, fd_degree_dyadic) and makes the
eigensolver entry points return FD_ERR_INVALID_ARG before any other work; a
later call on clean data through the same workspace is unaffected.  The same
holds for float32 X whose beta log2(e) max ||x - mean||^2 is beyond 65488,
where the float16 offset pieces cannot hold the exponent: NaN outputs, or
FD_ERR_UNSUPPORTED from the eigensolver and continuation, and the flow stops
its sweep there (exit reason "range").  A warm start whose columns repeat
(rank-deficient) or vanish is completed by the solver's orthonormalisation,
and the eigenvalues equal a cold solve's.
"""
import os
import subprocess

import numpy as np
import pytest
import torch

from gpu_util import TOL_F32, case, device, rel_fro, to_dev, to_np
from oracle import eig as oe
from oracle import kernel as ok
from paper_2609_38198_amd import _lib as fd
from paper_2609_38198_amd import inputs

pytestmark = pytest.mark.gpu


def _poisoned(X, i, f, value):
    Y = X.copy()
    Y[i, f] = value
    return Y


def test_product_nan_in_rows_or_columns_gives_nan_then_recovers():
    w = inputs.torus2()
    X = w.X
    dev = device()
    V = to_dev(inputs.random_block(w.N, 8), dev)
    ws = torch.empty(fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, w.N, w.N, w.D, 8),
                     dtype=torch.uint8, device=dev)
    case("non-finite: product with a NaN point")
    Y = to_np(fd.fd_kernel_matmul(to_dev(_poisoned(X, 77, 2, np.nan), dev), None, 8.0, V, ws=ws))
    assert np.isnan(Y).all()
    case("non-finite: rectangular product, +inf in the columns only")
    Xr = to_dev(X[:1000], dev)
    Xc = to_dev(_poisoned(X, 5, 0, np.inf), dev)
    Y = to_np(fd.fd_kernel_matmul(Xr, Xc, 8.0, V))
    assert np.isnan(Y).all()
    case("non-finite: clean product through the same workspace")
    Y = to_np(fd.fd_kernel_matmul(to_dev(X, dev), None, 8.0, V, ws=ws))
    ref = ok.kernel_matmul(X, None, 8.0, to_np(V))
    assert rel_fro(Y, ref) <= TOL_F32


def test_degree_nan_gives_nan():
    w = inputs.torus2()
    dev = device()
    case("non-finite: fd_degree with a NaN point")
    deg = fd.fd_degree(to_dev(_poisoned(w.X, 1, 1, np.nan), dev), 8.0, 0.5)
    for t in (deg.q, deg.d, deg.s, deg.s_off):
        assert np.isnan(to_np(t)).all()
    case("non-finite: fd_degree_dyadic with -inf")
    lad = fd.fd_degree_dyadic(to_dev(_poisoned(w.X, 2047, 3, -np.inf), dev), 0.5, 3, 0.5)
    for t in (lad.q, lad.d, lad.s, lad.s_off):
        assert np.isnan(to_np(t)).all()


def test_eigensolvers_refuse_non_finite_x():
    w = inputs.torus2()
    dev = device()
    Xbad = to_dev(_poisoned(w.X, 100, 0, np.nan), dev)
    case("non-finite: fd_block_lanczos refuses")
    with pytest.raises(fd.FdError) as e:
        fd.fd_block_lanczos(Xbad, 8.0, 8, 8)
    assert e.value.status == 1 and "NaN" in e.value.msg
    case("non-finite: fd_continuation refuses")
    with pytest.raises(fd.FdError) as e:
        fd.fd_continuation(Xbad, [1024, 2048], [8.0, 8.0], 8, 8)
    assert e.value.status == 1
    case("non-finite: fd_beta_flow refuses (bfloat16 NaN pattern)")
    bits = inputs.f32_to_bf16_bits(w.X)
    bits[10, 1] = 0x7FC0
    with pytest.raises(fd.FdError) as e:
        fd.fd_beta_flow(to_dev(bits, dev), 4, 8)
    assert e.value.status == 1


def clustered_points(seed=3, groups=24, per=6):
    # 144 points in tight clusters far apart: max ||x - mean||^2 = 210, so
    # beta = 100 is inside the exponent range (B = 3.0e4) and 1e4 beyond it
    rng = np.random.default_rng(seed)
    centres = rng.normal(size=(groups, 3)) * 4.0
    X = np.repeat(centres, per, axis=0) + rng.normal(size=(groups * per, 3)) * 0.3
    return (X - X.mean(0)).astype(np.float32)


def chain_points(n=200):
    # unit spacing on a line: max ||x - mean||^2 = 9900, so beta = 3 is inside
    # the range (B = 4.3e4, neighbours still coupled by e^-3) and 6 beyond it
    X = np.zeros((n, 3), dtype=np.float32)
    X[:, 0] = np.arange(n) - (n - 1) / 2
    return X


def test_exponent_range_async_entry_points_give_nan():
    X = clustered_points()
    dev = device()
    tX = to_dev(X, dev)
    V = to_dev(inputs.random_block(X.shape[0], 4), dev)
    case("exponent range: product inside (beta 100) is finite, beyond (1e4) NaN")
    assert np.isfinite(to_np(fd.fd_kernel_matmul(tX, None, 100.0, V))).all()
    assert np.isnan(to_np(fd.fd_kernel_matmul(tX, None, 1e4, V))).all()
    case("exponent range: rectangular product beyond the range")
    assert np.isnan(to_np(fd.fd_kernel_matmul(to_dev(X[:50], dev), tX, 1e4, V))).all()
    case("exponent range: fd_degree inside and beyond")
    deg = fd.fd_degree(tX, 100.0, 0.5)
    assert all(np.isfinite(to_np(t)).all() for t in (deg.q, deg.d, deg.s, deg.s_off))
    deg = fd.fd_degree(tX, 1e4, 0.5)
    for t in (deg.q, deg.d, deg.s, deg.s_off):
        assert np.isnan(to_np(t)).all()
    case("exponent range: fd_degree_dyadic whose last level is beyond")
    lad = fd.fd_degree_dyadic(tX, 100.0, 2, 0.5)
    assert np.isfinite(to_np(lad.q)).all()
    lad = fd.fd_degree_dyadic(tX, 100.0, 8, 0.5)
    for t in (lad.q, lad.d, lad.s, lad.s_off):
        assert np.isnan(to_np(t)).all()
    case("coordinate scale: huge coordinates at tiny bandwidths match the oracle")
    # B = 0.3 in both; the coordinate scale stays balanced (2^-24, 2^-34), so
    # neither side's float16 pieces lose bits
    for scale, beta in ((1e6, 1e-15), (1e9, 1e-21)):
        Xs = (X.astype(np.float64) * scale).astype(np.float32)
        Ys = to_np(fd.fd_kernel_matmul(to_dev(Xs, dev), None, beta, V))
        assert rel_fro(Ys, ok.kernel_matmul(Xs, None, beta, to_np(V))) <= TOL_F32
    case("exponent range: bfloat16 X has no such limit")
    Xb = to_dev(inputs.f32_to_bf16_bits(X), dev)
    assert np.isfinite(to_np(fd.fd_kernel_matmul(Xb, None, 1e4, V))).all()


def test_exponent_range_sync_entry_points_refuse():
    X = clustered_points()
    tX = to_dev(X, device())
    case("exponent range: fd_block_lanczos refuses beyond the range")
    with pytest.raises(fd.FdError) as e:
        fd.fd_block_lanczos(tX, 1e4, 4, 4)
    assert e.value.status == 2 and "exponent range" in e.value.msg
    case("exponent range: fd_continuation refuses at the first step beyond")
    with pytest.raises(fd.FdError) as e:
        fd.fd_continuation(tX, [144, 144], [100.0, 1e4], 4, 4, allow=(0, 5))
    assert e.value.status == 2 and "exponent range" in e.value.msg
    case("exponent range: fd_beta_flow whose first bandwidth is beyond")
    got = fd.fd_beta_flow(tX, 4, 4, fopts=fd.flow_default_opts(beta_start=1e4, max_probes=4),
                          allow=(2,))
    assert got.status == 2 and got.reason == "range" and len(got.probes) == 0


def test_flow_stops_at_the_exponent_range():
    X = chain_points()
    case("exponent range: flow on a 200-point chain from beta 3 (6 is beyond)")
    got = fd.fd_beta_flow(to_dev(X, device()), 4, 4,
                          fopts=fd.flow_default_opts(beta_start=3.0, max_probes=4), allow=(0, 5))
    assert got.reason == "range"
    assert [p["beta"] for p in got.probes] == [3.0]
    assert got.beta_x == 3.0 and got.probes[0]["admissible"]


JACOBI_CHECK = os.path.join(os.path.dirname(os.path.abspath(__file__)), "capi", "jacobi_check")


def test_dense_eigensolve_sorts_nan_last():
    # the Rayleigh-Ritz eigensolve on matrices with NaN on the diagonal (one
    # workgroup at m = 100, block Jacobi at m = 300): it finishes and returns
    # every number, descending, before the NaNs (tests/capi/jacobi_check.cpp)
    case("jacobi_eig with NaN diagonals, m = 100 and 300")
    assert os.path.exists(JACOBI_CHECK), "jacobi_check is not built (run __graft_entry__.build())"
    res = subprocess.run([JACOBI_CHECK], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.count("order ok") == 2, res.stdout


@pytest.mark.parametrize("kind", ["duplicate", "zero"])
def test_rank_deficient_warm_start(kind):
    # k = 16 pairs of the 2-torus; the warm start repeats each of 8 Markov
    # vectors twice, or is all zeros: the solver replaces the dependent
    # columns and converges to the cold solve's eigenvalues
    w = inputs.torus2()
    dev = device()
    tX = to_dev(w.X, dev)
    k, b, beta = 16, 8, 8.0
    sp = oe.spectrum(w.X, beta, 0.5, k + 4)
    if kind == "duplicate":
        half = sp.psi[:, :8].astype(np.float32)
        V0 = np.repeat(half, 2, axis=1)
    else:
        V0 = np.zeros((w.N, k), dtype=np.float32)
    case(f"rank-deficient warm start ({kind}) torus2 k=16 b=8")
    e = fd.fd_block_lanczos(tX, beta, k, b, V0=to_dev(np.ascontiguousarray(V0), dev))
    ev = np.asarray(e.evals)
    assert e.info["nconv"] == k
    assert np.all(np.abs(ev - sp.evals[:k]) <= np.maximum(1e-5 * np.abs(sp.evals[:k]), 1e-6))
    phi = to_np(e.evecs)
    assert np.abs(phi.T @ phi - np.eye(k)).max() <= 1e-5
