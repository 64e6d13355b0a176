"""fd_continuation: warm-started (n, beta) ladder, Nystrom extension, Perron wall.

Every step's eigenvalues must equal the oracle's dense eigensolve on the same
prefix at the same beta (a warm start may change the work, never the answer),
and the Markov vectors of the final step must span the oracle's leading
invariant subspaces.  The wall flag must agree with the oracle's Perron gap
g_P <= kappa_P * eta_fp32 = 1e-6 (Sec. 2.3, eq. perronwall).
"""
import numpy as np
import pytest

from gpu_util import case, device, to_dev, to_np
from oracle import diagnostics as od
from oracle import kernel as ok
from oracle import eig as oe
from paper_2609_38198_amd import _lib as fd
from paper_2609_38198_amd import inputs

pytestmark = pytest.mark.gpu


def eval_ok(got, ref):
    got = np.asarray(got)
    ref = np.asarray(ref)
    return np.all(np.abs(got - ref) <= np.maximum(1e-5 * np.abs(ref), 1e-6))


def test_ladder_matches_cold_solves():
    w = inputs.torus2()
    X = w.X
    ns = [512, 512, 1024, 1024, 2048, 2048]
    bs = [2.0, 4.0, 2.0, 4.0, 2.0, 4.0]
    k, b = 8, 8
    dev = device()
    tX = to_dev(X, dev)
    case("continuation torus2 ladder 512->2048, beta 2/4")
    lad = fd.fd_continuation(tX, ns, bs, k, b)
    assert lad.steps_done == len(ns)
    for t, (n, beta) in enumerate(zip(ns, bs)):
        sp = oe.spectrum(X[:n], beta, 0.5, k + 4)
        assert eval_ok(lad.evals[t], sp.evals[:k]), (t, lad.evals[t], sp.evals[:k])
        assert lad.info[t]["nconv"] == k
    sp = oe.spectrum(X, bs[-1], 0.5, k + 4)
    psi = to_np(lad.psi)
    cuts = [c for c in range(1, k) if sp.evals[c - 1] - sp.evals[c] >= 1e-2]
    for c in cuts:
        assert od.principal_angles(psi[:, :c], sp.psi[:, :c]).max() < 1e-3
    # a warm start never costs more products than a cold solve of the same step
    cold = fd.fd_block_lanczos(tX, bs[-1], k, b)
    print("matvecs per step", [i["block_matvecs"] for i in lad.info], "cold", cold.info["block_matvecs"])
    assert lad.info[-1]["block_matvecs"] <= cold.info["block_matvecs"]


def test_nystrom_step_starts_close():
    # after the prefix doubles, the extended start is a valid basis: the step
    # reaches the dense eigenvalues and needs no more products than a cold
    # solve at that size
    X = inputs.torus_points(4096, 2, seed=3).astype(np.float32)
    dev = device()
    tX = to_dev(X, dev)
    case("continuation Nystrom 2048 -> 4096 at beta 2")
    lad = fd.fd_continuation(tX, [2048, 4096], [2.0, 2.0], 8, 8)
    cold = fd.fd_block_lanczos(tX, 2.0, 8, 8)
    sp = oe.spectrum(X, 2.0, 0.5, 12)
    assert eval_ok(lad.evals[1], sp.evals[:8])
    print("nystrom step", lad.info[1]["block_matvecs"], "cold", cold.info["block_matvecs"])
    assert lad.info[1]["nconv"] == 8
    assert lad.info[1]["block_matvecs"] <= cold.info["block_matvecs"]


def test_wall_flag_and_stop():
    wl = inputs.torus6_noisy(N=4096)
    X = wl.X
    gaps = {}
    for beta in (2.0, 8.0):
        sp = oe.spectrum(X, beta, 0.5, 4)
        gaps[beta] = od.perron_gap(sp.evals)
    assert od.wall_admissible(gaps[2.0], "fp32") and not od.wall_admissible(gaps[8.0], "fp32")
    dev = device()
    case("continuation wall noisy 6-torus N=4096 beta 2 -> 8 -> 16")
    lad = fd.fd_continuation(to_dev(X, dev), [4096, 4096, 4096], [2.0, 8.0, 16.0], 4, 8,
                             stop_at_wall=True, allow=(0, 6))
    assert lad.status == 6
    assert lad.steps_done == 2
    assert lad.info[0]["wall"] == 0 and lad.info[1]["wall"] == 1
    assert lad.info[0]["gap_perron"] == pytest.approx(gaps[2.0], rel=1e-3)


def test_noisy_torus6_ladder_at_its_sizes():
    # the noisy 6-torus ladder with the default options: n in {16384, 65536,
    # 262144} x beta doubling 0.5 -> 8, k = 64, b = 32, each step warm-started
    # from the previous one (Nystrom extension when n grows).  Every step short
    # of the Perron wall converges all 64 pairs; (16384, 8) is at the wall
    # (g_P ~ 9e-7 <= kappa_P eta_fp32); the final step's Ritz pairs are true
    # eigenpairs of the exact operator on sampled rows, and a warm step's
    # eigenvalues equal a cold solve's
    w = inputs.torus6_noisy()
    X = w.X
    ns = [n for n in w.extra["n_ladder"] for _ in w.betas]
    bs = [beta for _ in w.extra["n_ladder"] for beta in w.betas]
    k, b = w.k, w.b
    dev = device()
    tX = to_dev(X, dev)
    case("continuation noisy 6-torus ladder 16384 / 65536 / 262144 x beta 0.5 .. 8, k=64 b=32")
    lad = fd.fd_continuation(tX, ns, bs, k, b, opts=fd.default_opts(verbose=1))
    assert lad.status == 0 and lad.steps_done == len(ns)
    for t, (n, beta) in enumerate(zip(ns, bs)):
        i = lad.info[t]
        print(f"n={n} beta={beta}: products {i['block_matvecs']}, nconv {i['nconv']}, "
              f"gap {i['gap_perron']:.3e}, wall {i['wall']}, {i['seconds']:.2f} s")
        if (n, beta) == (16384, 8.0):
            assert i["wall"] == 1 and i["gap_perron"] <= 1e-6
        else:
            assert i["wall"] == 0 and i["gap_perron"] > 1e-6
            assert i["nconv"] == k and i["max_residual"] <= 1e-5
    # the final step (262144, 8): residuals with the exact operator on 48 rows
    n, beta = ns[-1], bs[-1]
    phi = to_np(lad.evecs)
    theta = np.asarray(lad.evals[-1])
    deg = fd.fd_degree(tX[:n], beta, 0.5)
    q, s = to_np(deg.q), to_np(deg.s)
    X64 = X[:n].astype(np.float64)
    rows = np.random.default_rng(31).choice(n, 48, replace=False)
    ones = np.ones((n, 1))
    q_ref = ok.kernel_matmul(X64, None, beta, ones, rows=rows, threads=8)[:, 0]
    assert np.linalg.norm(q[rows] - q_ref) <= 1e-5 * np.linalg.norm(q_ref)
    mphi = ok.kernel_matmul(X64, None, beta, phi, sl=s, sr=s, rows=rows, threads=8)
    r = mphi - phi[rows] * theta[None, :]
    print(f"final step: max |M phi - theta phi| on sampled rows {np.abs(r).max():.2e}")
    assert np.abs(r).max() <= 1.5e-5
    assert np.abs(phi.T @ phi - np.eye(k)).max() <= 1e-5
    # warm == cold at (16384, 2)
    t2 = ns.index(16384) + list(w.betas).index(2.0)
    case("cold solve n=16384 beta=2 k=64 b=32")
    cold = fd.fd_block_lanczos(tX[:16384], 2.0, k, b)
    assert eval_ok(lad.evals[t2], cold.evals), (np.abs(np.asarray(lad.evals[t2]) -
                                                       np.asarray(cold.evals)).max())
