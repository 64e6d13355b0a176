"""The library's host-side decision logic on the CPU, under the address and
undefined-behaviour sanitizers: the eigensolver's layout, check schedule,
convergence count, restart block and Perron-wall stop, the continuation's
Nystrom source, and the beta flow's sweep (Sec. 2.3) over mocked probes,
compared probe by probe with the oracle's flow on the same mocks."""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import beta_flow as bf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "host", "host_logic_check.cpp")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    out = str(tmp_path_factory.mktemp("hostlogic") / "host_logic_check")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-Wall", "-Wextra", "-Werror",
           "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2609_38198_amd", "csrc"), SRC, "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    return out


def _env():
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


def test_solver_and_continuation_bookkeeping(driver):
    res = subprocess.run([driver, "units"], capture_output=True, text=True, env=_env())
    assert res.returncode == 0, res.stdout + res.stderr
    assert "0 failures" in res.stdout


def run_flow(driver, N, beta0, max_probes, vb, soff, gaps, dtype="fp32", k=4):
    eta = {"fp32": 1e-7, "bf16": 8e-3}[dtype]
    spec = [f"{N} {beta0!r} {max_probes} {eta!r} 10.0 6.0 {k} 0 {len(vb)}"]
    spec += [f"{float(a)!r} {float(b)!r} {float(c)!r}" for a, b, c in zip(vb, soff, gaps)]
    res = subprocess.run([driver, "flow"], input="\n".join(spec) + "\n", capture_output=True,
                         text=True, env=_env())
    assert res.returncode == 0, res.stderr
    recs, outcome = [], None
    for line in res.stdout.splitlines():
        f = line.split()
        if f[0] == "record":
            rec = dict(role=int(f[2]), beta=float(f[3]), s_off=float(f[4]), gap=float(f[5]),
                       v_bias=float(f[6]), v_mach=float(f[7]), n_eff=float(f[8]),
                       v_stat=float(f[9]), v_total=float(f[10]), d_hat=float(f[11]),
                       admissible=bool(int(f[12])))
            if int(f[1]):
                recs[-1] = rec
            else:
                recs.append(rec)
        elif f[0] == "outcome":
            outcome = dict(any=bool(int(f[1])), reason=int(f[2]), beta_x=float(f[3]))
    return recs, outcome


def oracle_mock(vb, soff, gaps, beta0, dtype="fp32"):
    def probe(beta):
        i = max(0, min(int(round(math.log2(beta / beta0))), len(vb) - 1))
        ev = np.array([1.0, 1.0 - gaps[i], math.exp(-vb[i]), math.exp(-vb[i])])
        return bf.make_probe(beta, ev, soff[i], dtype)
    return probe


REASON = {0: "bracket", 1: "wall", 2: "budget"}


def compare(driver, N, beta0, max_probes, vb, soff, gaps, dtype="fp32"):
    recs, out = run_flow(driver, N, beta0, max_probes, vb, soff, gaps, dtype)
    ref = bf.flow(oracle_mock(vb, soff, gaps, beta0, dtype), N, beta0, max_probes=max_probes)
    dyadic = [r for r in recs if r["role"] == 0 and r["admissible"]]
    assert len(dyadic) == len(ref.probes)
    for g, r in zip(dyadic, ref.probes):
        assert g["beta"] == pytest.approx(r.beta, rel=1e-15)
        assert g["gap"] == pytest.approx(r.gap, rel=1e-12)
        assert g["v_bias"] == pytest.approx(r.v_bias, rel=1e-12)
        assert g["v_mach"] == pytest.approx(r.v_mach, rel=1e-12)
        if r.v_total is None:
            assert math.isnan(g["v_total"])
        else:
            assert g["n_eff"] == pytest.approx(r.n_eff, rel=1e-12)
            assert g["v_stat"] == pytest.approx(r.v_stat, rel=1e-12)
            assert g["v_total"] == pytest.approx(r.v_total, rel=1e-12)
            assert g["d_hat"] == pytest.approx(r.d_hat, rel=1e-12, abs=1e-12)
    assert REASON[out["reason"]] == ref.reason
    if ref.probes:
        assert out["any"] and out["beta_x"] == pytest.approx(ref.beta_x, rel=1e-12)
    else:
        assert not out["any"]
    return out


def test_flow_bracket_wall_budget_like_the_oracle(driver):
    N = 1000
    vb = [4.0, 2.0, 1.0, 0.5, 0.25, 0.12, 0.06]
    soff = [N * 400 / 2 ** i for i in range(4)] + [N * 400 / 2 ** 3 / 8 ** j for j in range(1, 4)]
    assert REASON[compare(driver, N, 0.1, 7, vb, soff, [0.5] * 7)["reason"]] == "bracket"
    gaps = [0.5, 0.2, 1e-3, 2e-5, 1e-7, 1e-8, 1e-8]
    assert REASON[compare(driver, N, 0.1, 6, vb, soff, gaps)["reason"]] == "wall"
    assert REASON[compare(driver, N, 0.1, 4, vb[:4], soff[:4], [0.5] * 4)["reason"]] == "budget"
    # bfloat16 eta: the wall comes at g_P <= 0.08
    gaps = [0.5, 0.3, 0.05, 0.02, 0.01, 0.01, 0.01]
    assert REASON[compare(driver, N, 0.1, 7, vb, soff, gaps, "bf16")["reason"]] == "wall"
    # the first probe already past the wall: nothing admissible
    assert not compare(driver, N, 0.1, 5, vb, soff, [1e-9] * 7)["any"]


@pytest.mark.parametrize("seed", range(24))
def test_flow_random_sequences_like_the_oracle(driver, seed):
    # random mocked sweeps: V_bias halving with noise, S_off falling at a
    # random rate, Perron gaps shrinking towards the wall
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 10))
    N = int(rng.integers(100, 100000))
    vb = list(4.0 * np.cumprod(rng.uniform(0.35, 0.7, n)))
    soff = list(N * 500.0 * np.cumprod(rng.uniform(0.05, 0.8, n)))
    gaps = list(0.9 * np.cumprod(rng.uniform(1e-3, 0.6, n)))
    compare(driver, N, float(rng.uniform(0.01, 1.0)), int(rng.integers(2, n + 2)), vb, soff,
            gaps, "bf16" if seed % 5 == 0 else "fp32")
