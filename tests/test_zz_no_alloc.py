"""The allocation-free product (fd_kernel_matmul_noalloc): same bits as
fd_kernel_matmul with a workspace, and the oracle's values to the float32
bar, on consecutive calls whose second input is smaller than the first; a
problem too large for the built-in scratch is refused."""
import numpy as np
import pytest
import torch

from gpu_util import TOL_BF16, TOL_F32, case, device, rel_fro, to_dev, to_np
from oracle import kernel as ok
from paper_2609_38198_amd import _lib as fd
from paper_2609_38198_amd import inputs

pytestmark = pytest.mark.gpu


def _points(N, D, seed, scale=0.5):
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(N, D)) * scale
    return (X - X.mean(0)).astype(np.float32)


def _both(X, Xc_rows, beta, V, sl, sr):
    """(no-alloc result, workspace result) for rows X and columns X[:Xc_rows]."""
    dev = device()
    tX = to_dev(X, dev)
    tXc = tX if Xc_rows is None else tX[:Xc_rows]
    tV = to_dev(V, dev)
    tsl = None if sl is None else to_dev(sl, dev)
    tsr = None if sr is None else to_dev(sr, dev)
    Y0 = torch.full((X.shape[0], V.shape[1]), float("nan"), dtype=torch.float32, device=dev)
    fd.fd_kernel_matmul_noalloc(tX, tXc, beta, tV, Y0, sl=tsl, sr=tsr)
    Y1 = fd.fd_kernel_matmul(tX, tXc, beta, tV, sl=tsl, sr=tsr)
    torch.cuda.synchronize()
    return Y0, Y1


def test_consecutive_calls_match_the_workspace_entry_point():
    # call 1: 20,000 points in R^12 (ragged against every tile size), b = 16,
    # both scales; call 2: a smaller, rectangular problem in R^30 with b = 32
    # (columns a prefix of the rows) right after it on the same scratch
    N1, D1, b1, beta1 = 20000, 12, 16, 2.0
    X1 = _points(N1, D1, 1)
    V1 = inputs.random_block(N1, b1, seed=11)
    rng = np.random.default_rng(2)
    sl1 = rng.uniform(0.5, 2.0, N1).astype(np.float32)
    sr1 = rng.uniform(0.5, 2.0, N1).astype(np.float32)
    case(f"no-alloc call 1: N={N1} D={D1} b={b1} beta={beta1}")
    Y0, Y1 = _both(X1, None, beta1, V1, sl1, sr1)
    assert torch.equal(Y0, Y1)
    rows = np.random.default_rng(3).choice(N1, 256, replace=False)
    ref = ok.kernel_matmul(X1, None, beta1, V1, sl=sl1, sr=sr1, rows=rows, threads=8)
    assert rel_fro(to_np(Y0)[rows], ref) <= TOL_F32

    N2, Nc2, D2, b2 = 3001, 1777, 30, 32
    X2 = _points(N2, D2, 4, scale=0.3)
    beta2 = 1.0 / (D2 * 0.09)
    V2 = inputs.random_block(Nc2, b2, seed=12)
    case(f"no-alloc call 2: Nr={N2} Nc={Nc2} D={D2} b={b2} beta={beta2:.4f}")
    Y0, Y1 = _both(X2, Nc2, beta2, V2, None, None)
    assert torch.equal(Y0, Y1)
    ref = ok.kernel_matmul(X2, X2[:Nc2], beta2, V2, threads=8)
    assert rel_fro(to_np(Y0), ref) <= TOL_F32


def test_single_column_and_bf16():
    # b = 1 (the row-sum path) and bfloat16 points, each against the workspace
    # entry point bit for bit and against the oracle
    N, D = 4099, 8
    X = _points(N, D, 5)
    v = inputs.random_block(N, 1, seed=13)
    case(f"no-alloc b=1 N={N} D={D}")
    Y0, Y1 = _both(X, None, 1.5, v, None, None)
    assert torch.equal(Y0, Y1)
    assert rel_fro(to_np(Y0), ok.kernel_matmul(X, None, 1.5, v, threads=8)) <= TOL_F32

    N, D, b = 2500, 64, 64
    bits = inputs.f32_to_bf16_bits(_points(N, D, 6, scale=0.2))
    V = inputs.random_block(N, b, seed=14)
    beta = 1.0 / (D * 0.08)
    case(f"no-alloc bf16 N={N} D={D} b={b}")
    Y0, Y1 = _both(bits, None, beta, V, None, None)
    assert torch.equal(Y0, Y1)
    ref = ok.kernel_matmul(inputs.bf16_bits_to_f64(bits), None, beta, V, threads=8)
    assert rel_fro(to_np(Y0), ref) <= TOL_BF16


def test_too_large_is_refused_before_any_work():
    dev = device()
    N, D, b = 1 << 20, 30, 32
    X = torch.empty((N, D), dtype=torch.float32, device=dev)
    V = torch.empty((N, b), dtype=torch.float32, device=dev)
    Y = torch.empty((N, b), dtype=torch.float32, device=dev)
    assert fd.fd_kernel_matmul_noalloc_limit() == 256 << 20
    case("no-alloc refusal N=2^20 D=30 b=32")
    with pytest.raises(fd.FdError) as e:
        fd.fd_kernel_matmul_noalloc(X, None, 1.0, V, Y)
    assert e.value.status == 3  # FD_ERR_WORKSPACE
