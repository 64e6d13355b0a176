"""The C ABI driven from C++ alone: tests/capi/capi_check (built with the
library) runs fd_degree, a normalised fd_kernel_matmul and fd_block_lanczos on
device buffers it allocates itself, plus one rejected call; its outputs are
checked here against the oracle to the same bars as the Python-side tests.
"""
import os
import subprocess

import numpy as np
import pytest

from gpu_util import case
from oracle import diagnostics as od
from oracle import eig as oe
from oracle import kernel as ok
from oracle import normalise as on

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "capi", "capi_check")


def run_capi(tmp_path, X, V, b, k, beta, alpha):
    N, D = X.shape
    src = tmp_path / "in.bin"
    dst = tmp_path / "out.bin"
    with open(src, "wb") as fh:
        fh.write(np.ascontiguousarray(X, dtype=np.float32).tobytes())
        fh.write(np.ascontiguousarray(V, dtype=np.float32).tobytes())
    assert os.path.exists(EXE), "capi_check is not built (run __graft_entry__.build())"
    res = subprocess.run([EXE, str(N), str(D), str(b), str(k), repr(beta), repr(alpha), str(src),
                          str(dst)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, (res.returncode, res.stdout, res.stderr)
    raw = dst.read_bytes()
    out, pos = {}, 0

    def take(name, dtype, count):
        nonlocal pos
        nbytes = np.dtype(dtype).itemsize * count
        out[name] = np.frombuffer(raw[pos:pos + nbytes], dtype=dtype)
        pos += nbytes

    take("q", np.float32, N)
    take("d", np.float32, N)
    take("s", np.float32, N)
    take("s_off", np.float64, 1)
    take("Y", np.float32, N * b)
    take("evals", np.float64, k)
    take("res", np.float64, k)
    take("evecs", np.float32, N * k)
    take("tail", np.int32, 6)
    assert pos == len(raw)
    out["Y"] = out["Y"].reshape(N, b)
    out["evecs"] = out["evecs"].reshape(N, k)
    return out


def rel(a, b):
    return float(np.linalg.norm(np.asarray(a, np.float64) - b) / np.linalg.norm(b))


def test_c_abi_from_cpp(tmp_path):
    rng = np.random.default_rng(2609)
    N, D, b, k, beta, alpha = 700, 5, 8, 6, 1.5, 0.5
    X = rng.normal(size=(N, D))
    X = (X - X.mean(0)).astype(np.float32)
    V = rng.normal(size=(N, b)).astype(np.float32)
    case(f"capi_check N={N} D={D} b={b} k={k}")
    g = run_capi(tmp_path, X, V, b, k, beta, alpha)
    Xd = X.astype(np.float64)
    nrm = on.normalise(Xd, beta, alpha)
    assert rel(g["q"], nrm.q) <= 1e-5
    assert rel(g["d"], nrm.d) <= 1e-5
    assert rel(g["s"], nrm.s) <= 1e-5
    assert abs(g["s_off"][0] - nrm.s_off) <= 1e-5 * nrm.s_off
    ref = ok.kernel_matmul(Xd, None, beta, V.astype(np.float64), sl=nrm.s, sr=nrm.s)
    assert rel(g["Y"], ref) <= 1e-5
    restarts, matvecs, nconv, status, bad, msg_len = (int(v) for v in g["tail"])
    assert status == 0 and nconv == k and matvecs > 0
    sp = oe.spectrum(Xd, beta, alpha, k + 4)
    tol = np.maximum(1e-5 * np.abs(sp.evals[:k]), 1e-6)
    assert np.all(np.abs(g["evals"] - sp.evals[:k]) <= tol), (g["evals"], sp.evals[:k])
    phi = g["evecs"].astype(np.float64)
    assert np.abs(phi.T @ phi - np.eye(k)).max() <= 1e-5
    assert g["res"].max() <= 1e-5
    cuts = [c for c in range(1, k) if sp.evals[c - 1] - sp.evals[c] >= 1e-2]
    for c in cuts:
        assert od.principal_angles(phi[:, :c], sp.phi[:, :c]).max() < 1e-3
    # the rejected call (block width 0): FD_ERR_INVALID_ARG with a message
    assert bad == 1 and msg_len > 0
