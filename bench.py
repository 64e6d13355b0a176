#!/usr/bin/env python3
"""Benchmark of the diffusion-map hot path on one MI355X.

One step = one pass of the path over the molecule-like workload (N = 2^20
points in R^30, float32, block width b = 32, alpha = 1/2, beta = 1 / median
squared distance of a 4,096-point subsample): the normalisation vectors
(q = K 1, w = q^-a, d = w (K w), s = w d^-1/2: two passes over the kernel,
`fd_degree`) and one fused normalised product Y = diag(s) K diag(s) V
(`fd_kernel_matmul`).  Inputs are resident in HBM before the timed region.

Printed value: whole-step throughput in kernel pair-columns per second,
N^2 * b divided by the step time (the normalisation passes are inside the
step time).  The roofline object is for the fused product, the kernel with
the larger share of the step, timed with HIP events on its launch stream.
Its bound is the transcendental rate: every kernel entry costs one
v_exp_f32, and the matrix-core work of the contractions does not run
concurrently with the vector ALUs on gfx950, so the exponentials set the
floor.  HBM traffic comes from the rocprofv3 counter summary under
profiles/ when that summary was taken on the current kernel sources, else
it is null.

Extra fields: `lanczos_top64_s`, the wall time of `fd_block_lanczos` to
the top 64 eigenpairs on the same workload (both normalisation passes
included), and `torus6_sweep`, the flat 6-torus sweep (N = 65,536, D = 12,
b = 16, beta in {0.5, 1, 2, 4, 8}: the dyadic normalisation ladder and one
normalised product per beta).  Optional legs add other workloads
(see --help).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
# v_exp_f32 issues a wave64 in 8 cycles (half the plain-VALU rate of 16
# lanes/cycle): 256 CUs x 4 SIMDs x 8 lanes x 2.4 GHz
PEAK_EXP_TS = 256 * 4 * 8 * 2.4e9 / 1e12
PEAK_F16_MFMA_TFS = 2516.6
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_molecule.md")
TRAFFIC_FILE_TORUS6 = os.path.join(ROOT, "profiles", "hbm_traffic_torus6.md")
CONTRACTION = ("exponent: float16 matrix instructions over three-piece float16 splits of the "
               "float32 coordinates (short split for D > 4 within its tested exponent budget, "
               "exact split otherwise), float32 accumulate; K V: float16 two-term splits of K "
               "and V, three float16 matrix instructions per 16 columns, float32 accumulate")
KERNEL_SOURCES = ("hx_kernels.hip", "kv_common.hpp", "kv_kernels.hip", "fd_internal.hpp")


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_38198_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel: str, path: str = TRAFFIC_FILE):
    """HBM bytes per launch of `kernel` from a counter summary, if current."""
    try:
        with open(path) as fh:
            text = fh.read()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        line = line.strip().lstrip("-* ")
        if ":" in line:
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    v = fields.get(f"{kernel}_hbm_bytes_per_launch")
    return float(v) if v else None


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(X: np.ndarray, beta: float, b: int, seconds: float, label: str) -> dict:
    """Time the oracle's product on a bounded sample of rows (float64, CPU)."""
    from oracle import kernel as ok
    from paper_2609_38198_amd import inputs

    cores = min(len(os.sched_getaffinity(0)), 16)
    N = X.shape[0]
    V = inputs.random_block(N, b, seed=2)
    rng = np.random.default_rng(0)
    # row blocks of 16 keep a thread's float64 temporaries near 256 MB at
    # N = 2^20; rounds of one block per thread run until the time is spent
    blk = 16 if N > (1 << 18) else 64
    order = rng.permutation(N)
    per_round = blk * cores
    nrows = 0
    t0 = time.perf_counter()
    while nrows + per_round <= N:
        rows = order[nrows:nrows + per_round]
        ok.kernel_matmul(X, None, beta, V, rows=rows, block=blk, threads=cores)
        nrows += per_round
        if time.perf_counter() - t0 >= seconds:
            break
    t = time.perf_counter() - t0
    return {"value": nrows * N * b / t, "unit": "pair-cols/s", "cores": cores, "kind": "oracle",
            "sample": f"{label}: float64 difference-form product K V on {nrows} seeded rows x "
                      f"all {N} columns, b={b}, beta={beta:.5g}, {t:.1f} s on {cores} threads "
                      f"of {cpu_model()}"}


def lanczos_leg(fd, torch, dev) -> dict:
    from paper_2609_38198_amd import inputs
    w = inputs.torus2()
    X = torch.from_numpy(w.X).to(dev)
    fd.fd_block_lanczos(X, w.betas[0], w.k, w.b)  # warm-up (code objects, allocator)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e = fd.fd_block_lanczos(X, w.betas[0], w.k, w.b)
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    return {"workload": "torus2 N=2048 D=4 beta=8 b=8 k=16", "seconds": t,
            "block_matvecs": e.info["block_matvecs"], "restarts": e.info["restarts"],
            "max_residual": e.info["max_residual"]}


def lanczos_top64_leg(fd, torch, w, X) -> dict:
    """Top-64 eigenpairs of the step's workload (molecule-like, N = 2^20, D = 30, b = 32)."""
    beta = float(w.betas[0])
    torch.cuda.synchronize()
    fd.fd_profile_read(fd.FD_KERNEL_PRODUCT)
    fd.fd_profile_read(fd.FD_KERNEL_ROWSUM)
    fd.fd_profile_enable(True)
    log(f"top-64 leg: N={w.N} beta={beta:.5f} start")
    t0 = time.perf_counter()
    e = fd.fd_block_lanczos(X, beta, w.k, w.b, allow_not_converged=True,
                            opts=fd.default_opts(verbose=1))
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    fd.fd_profile_enable(False)
    pms, pn = fd.fd_profile_read(fd.FD_KERNEL_PRODUCT)
    rms, rn = fd.fd_profile_read(fd.FD_KERNEL_ROWSUM)
    log(f"top-64 leg: {t:.3f} s, {e.info['block_matvecs']} block products, "
        f"{e.info['nconv']}/{w.k} converged")
    return {"seconds": t, "status": e.status, "block_matvecs": e.info["block_matvecs"],
            "restarts": e.info["restarts"], "nconv": e.info["nconv"],
            "max_residual": e.info["max_residual"], "gap_perron": e.info["gap_perron"],
            "product_total_s": pms * 1e-3, "product_launches": pn,
            "rowsum_total_s": rms * 1e-3, "rowsum_launches": rn,
            "evals_head": e.evals[:4], "evals_tail": e.evals[-2:]}


def torus6_sweep_leg(fd, torch, dev, steps: int, warmup: int = 2) -> dict:
    """The flat 6-torus sweep: dyadic normalisation ladder + one normalised product per beta."""
    from paper_2609_38198_amd import inputs
    wl = inputs.torus6()
    N, D, b = wl.N, wl.D, wl.b
    betas, alpha = wl.betas, wl.alpha
    X = torch.from_numpy(wl.X).to(dev)
    V = torch.from_numpy(inputs.random_block(N, b)).to(dev)
    Y = torch.empty((N, b), dtype=torch.float32, device=dev)
    ws_p = torch.empty(fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, N, N, D, b),
                       dtype=torch.uint8, device=dev)
    ws_d = torch.empty(fd.fd_workspace_size(fd.FD_OP_DEGREE_DYADIC, N, N, D),
                       dtype=torch.uint8, device=dev)
    nb = len(betas)
    # K at 2 beta is K at beta squared entrywise: each level's q comes from
    # the previous level's second pass
    assert all(betas[i + 1] == 2.0 * betas[i] for i in range(nb - 1))

    def step():
        lad = fd.fd_degree_dyadic(X, betas[0], nb, alpha, ws=ws_d)
        for l, beta in enumerate(betas):
            fd.fd_kernel_matmul(X, None, beta, V, sl=lad.s[l], sr=lad.s[l], Y=Y, ws=ws_p)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    fd.fd_profile_read(fd.FD_KERNEL_PRODUCT)
    fd.fd_profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t = (time.perf_counter() - t0) / steps
    fd.fd_profile_enable(False)
    pms, pn = fd.fd_profile_read(fd.FD_KERNEL_PRODUCT)
    avg = pms * 1e-3 / max(pn, 1)
    return {"workload": f"flat 6-torus N={N} D={D} b={b} beta sweep {list(betas)} "
                        f"alpha={alpha}", "steps": steps, "ms_per_step": t * 1e3,
            "pair_cols_per_s": nb * float(N) * N * b / t,
            "product_avg_ms": avg * 1e3, "product_texp_per_s": float(N) * N / avg / 1e12,
            "product_frac_exp_peak": float(N) * N / avg / 1e12 / PEAK_EXP_TS,
            "product_hbm_bytes_per_launch": recorded_traffic("product", TRAFFIC_FILE_TORUS6)}


def continuation_leg(fd, torch, dev, cold: bool = False) -> dict:
    """Noisy 6-torus ladder: n in {16K, 65K, 262K} x beta doubling 0.5 -> 8, k = 64, b = 32.

    cold: also solve every step from a random start (fd_block_lanczos on the
    prefix) and report its block products beside the warm-started ones.
    """
    from paper_2609_38198_amd import inputs
    w = inputs.torus6_noisy()
    X = torch.from_numpy(w.X).to(dev)
    ns, bs = [], []
    for n in w.extra["n_ladder"]:
        for beta in w.betas:
            ns.append(n)
            bs.append(beta)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    log("continuation leg: start")
    # default options: the steps at the Perron wall stop there and are
    # reported (wall = 1), every other step converges all 64 pairs
    opts = fd.default_opts(verbose=1)
    lad = fd.fd_continuation(X, ns, bs, w.k, w.b, allow=(0, 5), opts=opts)
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    steps = [{"n": n, "beta": beta, "matvecs": i["block_matvecs"], "nconv": i["nconv"],
              "gap": i["gap_perron"], "wall": i["wall"], "s": i["seconds"]}
             for n, beta, i in zip(ns, bs, lad.info)]
    if cold:
        log("continuation leg: cold solves of every step")
        for st in steps:
            t1 = time.perf_counter()
            e = fd.fd_block_lanczos(X[: st["n"]], st["beta"], w.k, w.b, alpha=0.5,
                                    opts=fd.default_opts(), allow_not_converged=True)
            torch.cuda.synchronize()
            st.update({"cold_matvecs": e.info["block_matvecs"], "cold_nconv": e.info["nconv"],
                       "cold_s": time.perf_counter() - t1})
            log(f"  n={st['n']} beta={st['beta']:g}: warm {st['matvecs']} / cold "
                f"{st['cold_matvecs']} block products")
    return {"workload": "noisy 6-torus N=262144 D=12 k=64 b=32, n in {16384, 65536, 262144} x "
                        "beta in {0.5, 1, 2, 4, 8}; default options", "seconds": t,
            "status": lad.status, "steps": steps}


def stress_leg(fd, torch, dev, iterations: int = 20) -> dict:
    """bfloat16 X, N = 2^21 in R^64: fused product throughput and 20 block-Lanczos iterations."""
    from paper_2609_38198_amd import inputs
    log("stress leg: generating N=2^21 x 64 bf16")
    w = inputs.stress()
    X = torch.from_numpy(w.X.view(np.int16)).to(dev).view(torch.bfloat16)
    N, D, b = w.N, w.D, w.b
    beta = float(w.betas[0])
    V = torch.from_numpy(inputs.random_block(N, b)).to(dev)
    Y = torch.empty((N, b), dtype=torch.float32, device=dev)
    ws = torch.empty(fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, N, N, D, b), dtype=torch.uint8,
                     device=dev)
    fd.fd_kernel_matmul(X, None, beta, V, Y=Y, ws=ws)
    torch.cuda.synchronize()
    fd.fd_profile_read(fd.FD_KERNEL_PRODUCT)
    fd.fd_profile_enable(True)
    reps = 3
    t0 = time.perf_counter()
    for _ in range(reps):
        fd.fd_kernel_matmul(X, None, beta, V, Y=Y, ws=ws)
    torch.cuda.synchronize()
    tp = (time.perf_counter() - t0) / reps
    fd.fd_profile_enable(False)
    pms, pn = fd.fd_profile_read(fd.FD_KERNEL_PRODUCT)
    del ws, Y
    avg = pms * 1e-3 / max(pn, 1)
    rec = {"workload": f"stress bf16 N={N} D={D} b={b} beta={beta:.5f}",
           "product_s": tp, "product_kernel_s": avg,
           "pair_cols_per_s": float(N) * N * b / avg,
           "exp_per_s": float(N) * N / avg}
    if iterations <= 0:
        return rec
    log(f"stress leg: product {tp:.3f} s; {iterations} block-Lanczos iterations")
    o = fd.default_opts(max_matvecs=iterations, max_basis_blocks=16, keep=64, verbose=1)
    t0 = time.perf_counter()
    e = fd.fd_block_lanczos(X, beta, 64, b, opts=o, allow_not_converged=True)
    torch.cuda.synchronize()
    tl = time.perf_counter() - t0
    rec.update({"lanczos_iters_s": tl, "iterations_cap": iterations,
                "block_matvecs": e.info["block_matvecs"], "nconv": e.info["nconv"],
                "max_residual": e.info["max_residual"], "evals_head": e.evals[:4],
                "evals_tail": e.evals[-2:]})
    return rec


# The paper's XGEMM timings for one raw kernel application K V on its T^6
# set-up (App. B, the matvec and matmat tables: fp32, D = 32, beta = 1, one
# RTX PRO 6000), seconds at N = 2^lg.  Context only: other hardware.
PAPER_XGEMM_S = {
    1: {16: 0.010897011, 18: 0.1407541988, 20: 2.08317415},
    8: {16: 0.012966476, 18: 0.152757719, 20: 2.897318638},
}


def paper_t6_leg(fd, torch, dev) -> dict:
    """Raw K V (b = 1 and 8) on the paper's T^6 set-up, beside its own timings."""
    from paper_2609_38198_amd import inputs
    rows = []
    for lg in (16, 18, 20):
        w = inputs.torus6_paper(1 << lg)
        N, D = w.N, w.D
        X = torch.from_numpy(w.X).to(dev)
        for b in (1, 8):
            V = torch.from_numpy(inputs.random_block(N, b)).to(dev)
            Y = torch.empty((N, b), dtype=torch.float32, device=dev)
            ws = torch.empty(fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, N, N, D, b),
                             dtype=torch.uint8, device=dev)
            fd.fd_kernel_matmul(X, None, 1.0, V, Y=Y, ws=ws)
            torch.cuda.synchronize()
            reps = 3 if lg >= 20 else 10
            t0 = time.perf_counter()
            for _ in range(reps):
                fd.fd_kernel_matmul(X, None, 1.0, V, Y=Y, ws=ws)
            torch.cuda.synchronize()
            t = (time.perf_counter() - t0) / reps
            paper = PAPER_XGEMM_S[b][lg]
            rows.append({"N": N, "b": b, "seconds": t, "pairs_per_s": float(N) * N / t,
                         "pair_cols_per_s": float(N) * N * b / t, "paper_xgemm_s": paper,
                         "paper_over_this": paper / t})
            del ws, Y, V
            log(f"paper T6 leg: N=2^{lg} b={b}: {t * 1e3:.2f} ms (paper {paper * 1e3:.2f} ms)")
    return {"workload": "anisotropic flat 6-torus, radii 1.00..1.50, D=32 zero-padded, beta=1, "
                        "seed 42, unnormalised K V", "rows": rows}


# The paper's one-GPU T^6 runs (Sec. 3, the data of figure t6scaling: fp32,
# k = 3 nontrivial modes, alpha = 1/2, one RTX PRO 6000): N -> (mean wall time
# s, its std, beta_x, its std, overlap score of the leading doublet).  Context
# only: other hardware, and the paper's timings include its own solver stack.
PAPER_T6_ONE_GPU = {
    1024: (6.0325, 4.5185, 0.36936, 0.03992, 0.92903),
    2048: (5.8926, 4.3790, 0.42356, 0.06325, 0.96819),
    4096: (5.8238, 4.4080, 0.49509, 0.08424, 0.98477),
    8192: (5.9655, 4.4799, 0.58220, 0.10710, 0.98515),
    16384: (6.3727, 4.9327, 0.68935, 0.13137, 0.99437),
    32768: (11.5528, 9.5942, 0.80013, 0.18802, 0.99428),
    65536: (15.9784, 10.9733, 0.91729, 0.27512, 0.99720),
    131072: (61.5799, 7.1353, 0.70902, 0.0, 0.99918),
    262144: (147.8957, 2.1209, 0.78405, 0.0, 0.99954),
    524288: (464.2531, 2.5314, 0.87415, 0.0, 0.99968),
    1048576: (2225.0375, 3.8461, 0.97949, 0.0, 0.99980),
}


def doublet_overlap(psi2: np.ndarray, theta_s: np.ndarray) -> float:
    """Recovery score of Sec. 3: overlap of the span of the leading two
    nontrivial Markov modes with span(cos theta_s, sin theta_s), both centred,
    in [0, 1]: the mean squared canonical correlation of the two planes
    (orthonormal bases by QR, float64)."""
    A = np.asarray(psi2, dtype=np.float64)
    B = np.stack([np.cos(theta_s), np.sin(theta_s)], 1)
    qa, _ = np.linalg.qr(A - A.mean(0))
    qb, _ = np.linalg.qr(B - B.mean(0))
    return float(np.sum((qa.T @ qb) ** 2) / 2.0)


def paper_t6_flow_leg(fd, torch, dev, max_lg: int) -> dict:
    """Sec. 3's solve on the paper's T^6 set-up: the beta flow with k = 3
    nontrivial modes (k = 4 with the Perron pair), alpha = 1/2, b = 8, from
    beta_0 of eq. beta0, at N = 2^10 .. 2^max_lg; time, beta_x and the
    doublet score beside the paper's one-GPU rows.  Repeats follow the
    paper's n_rep = clip(ceil(64^((22 - log2 N) / 12)), 1, 64), at most 8."""
    import math
    from paper_2609_38198_amd import inputs
    rows = []
    warm = inputs.torus6_paper(1024)
    fd.fd_beta_flow(torch.from_numpy(warm.X).to(dev), 4, 8, alpha=0.5)  # code objects
    torch.cuda.synchronize()
    for lg in range(10, max_lg + 1):
        N = 1 << lg
        w = inputs.torus6_paper(N)
        X = torch.from_numpy(w.X).to(dev)
        nrep = min(8, max(1, min(64, math.ceil(64 ** ((22 - lg) / 12)))))
        times, flow = [], None
        for _ in range(nrep):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            flow = fd.fd_beta_flow(X, 4, 8, alpha=0.5, allow=(0, 5))
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
        psi = flow.psi.double().cpu().numpy()
        score = doublet_overlap(psi[:, 1:3], w.extra["theta"][:, 5])
        p = PAPER_T6_ONE_GPU.get(N)
        row = {"N": N, "reps": nrep, "seconds": float(np.mean(times)),
               "seconds_std": float(np.std(times)), "beta_x": flow.beta_x,
               "exit": flow.reason, "probes": len(flow.probes), "status": flow.status,
               "evals": flow.evals, "overlap": score, "one_minus_overlap": 1.0 - score}
        if p is not None:
            row.update({"paper_seconds": p[0], "paper_seconds_std": p[1], "paper_beta_x": p[2],
                        "paper_beta_x_std": p[3], "paper_overlap": p[4],
                        "paper_over_this_time": p[0] / row["seconds"]})
        rows.append(row)
        log(f"paper T6 flow: N=2^{lg}: {row['seconds']:.3f} s x {nrep}, beta_x "
            f"{flow.beta_x:.4f} ({flow.reason}), 1 - overlap {1.0 - score:.2e}"
            + (f"; paper {p[0]:.1f} s, beta_x {p[2]:.3f}, 1 - overlap {1.0 - p[4]:.2e}"
               if p else ""))
        del X
    return {"workload": "paper T^6 (radii 1.00 .. 1.50, D = 32 zero-padded, seed 42): beta flow, "
                        "k = 3 nontrivial + Perron, alpha = 1/2, b = 8, fp32", "rows": rows}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-top64", action="store_true",
                    help="skip the top-64 eigensolve on the step's workload")
    ap.add_argument("--no-torus6", action="store_true", help="skip the flat 6-torus sweep")
    ap.add_argument("--only-torus6", action="store_true",
                    help="run only the flat 6-torus sweep (--steps / --warmup apply to it) and "
                         "print its record (for the counter runs of its kernels)")
    ap.add_argument("--lanczos", action="store_true",
                    help="time to the top 16 eigenpairs on the 2-torus (N = 2048)")
    ap.add_argument("--continuation", action="store_true")
    ap.add_argument("--continuation-cold", action="store_true",
                    help="with --continuation: also solve every ladder step from a random start")
    ap.add_argument("--stress", action="store_true",
                    help="bfloat16 stress set (N = 2^21, D = 64, b = 64): product throughput and "
                         "block-Lanczos iterations")
    ap.add_argument("--stress-iters", type=int, default=20,
                    help="block-Lanczos iterations of the stress leg (0: the product only)")
    ap.add_argument("--paper-t6", action="store_true",
                    help="raw K V on the paper's T^6 set-up (D=32, beta=1, b=1 and 8) beside "
                         "the paper's own timings")
    ap.add_argument("--paper-t6-flow", type=int, default=0, metavar="LOG2N",
                    help="Sec. 3's beta-flow solve on the paper's T^6 set-up at N = 2^10 .. "
                         "2^LOG2N beside the paper's one-GPU rows")
    ap.add_argument("--calibration-copy", type=int, default=0, metavar="MIB",
                    help="after the timed steps, copy MIB MiB device to device (a plain copy "
                         "kernel of known size, read by the HBM counter runs as their scale)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(row sharding is a design note, not code).", file=sys.stderr)
        return 2

    import torch

    from paper_2609_38198_amd import _lib as fd
    from paper_2609_38198_amd import inputs

    dev = torch.device("cuda:0")
    if args.only_torus6:
        rec = {"torus6_sweep": torus6_sweep_leg(fd, torch, dev, args.steps, args.warmup)}
        if args.calibration_copy > 0:
            src = torch.ones(args.calibration_copy << 18, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            dst.copy_(src)
            torch.cuda.synchronize()
            rec["calibration_copy_bytes"] = 2 * src.numel() * 4
        print(json.dumps(rec), flush=True)
        return 0
    log("generating the molecule-like workload (N = 2^20, D = 30)")
    wl = inputs.molecule()
    N, D, b = wl.N, wl.D, wl.b
    beta, alpha = float(wl.betas[0]), wl.alpha
    X = torch.from_numpy(wl.X).to(dev)
    V = torch.from_numpy(inputs.random_block(N, b)).to(dev)
    Y = torch.empty((N, b), dtype=torch.float32, device=dev)
    ws_p = torch.empty(fd.fd_workspace_size(fd.FD_OP_KERNEL_MATMUL, N, N, D, b),
                       dtype=torch.uint8, device=dev)
    ws_d = torch.empty(fd.fd_workspace_size(fd.FD_OP_DEGREE, N, N, D),
                       dtype=torch.uint8, device=dev)

    def step():
        deg = fd.fd_degree(X, beta, alpha, ws=ws_d)
        fd.fd_kernel_matmul(X, None, beta, V, sl=deg.s, sr=deg.s, Y=Y, ws=ws_p)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    fd.fd_profile_read(fd.FD_KERNEL_PRODUCT)
    fd.fd_profile_read(fd.FD_KERNEL_ROWSUM)
    fd.fd_profile_enable(True)
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    fd.fd_profile_enable(False)
    prod_ms, prod_n = fd.fd_profile_read(fd.FD_KERNEL_PRODUCT)
    row_ms, row_n = fd.fd_profile_read(fd.FD_KERNEL_ROWSUM)

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = float(N) * N * b / (ms_per_step * 1e-3)
    avg_prod_s = prod_ms * 1e-3 / max(prod_n, 1)
    avg_row_s = row_ms * 1e-3 / max(row_n, 1)
    # algorithmic work of one product launch: N^2 kernel entries (one
    # exponential each) and 2 N^2 (D + b) flops of the two contractions
    exp_prod = float(N) * N / avg_prod_s / 1e12
    flops = 2.0 * N * N * (D + b)
    # the row sums make the two normalisation applications (q = K 1, K w) in
    # two launches per step
    exp_row = float(N) * N / avg_row_s / 1e12
    log(f"step {ms_per_step:.1f} ms: product {avg_prod_s * 1e3:.1f} ms, "
        f"row-sum pass {avg_row_s * 1e3:.1f} ms")

    rec = {
        "metric": "fused K*V pair-cols/sec (N^2*b per sec)",
        "value": value,
        "unit": "pair-cols/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "contraction": CONTRACTION,
        "data": "synthetic",
        "config": {"workload": f"molecule-like manifold N={N} D={D} b={b} beta={beta:.5f} "
                               f"alpha={alpha}: normalisation vectors (2 passes) + 1 fused "
                               f"normalised product diag(s) K diag(s) V", "N": N, "D": D,
                   "b": b, "beta": beta, "alpha": alpha, "parallelism": "single GPU"},
        "roofline": {"bound": "alu", "kernel": "product", "achieved": exp_prod,
                     "peak": PEAK_EXP_TS, "unit": "Texp/s", "frac": exp_prod / PEAK_EXP_TS,
                     "traffic": recorded_traffic("product")},
        "roofline_mfma_f16": {"kernel": "product", "achieved": flops / avg_prod_s / 1e12,
                              "peak": PEAK_F16_MFMA_TFS, "unit": "TFLOP/s",
                              "frac": flops / avg_prod_s / 1e12 / PEAK_F16_MFMA_TFS,
                              "flops_per_launch": flops},
        "kernels": {
            "product": {"launches": prod_n, "avg_ms": avg_prod_s * 1e3,
                        "pair_cols_per_s": float(N) * N * b / avg_prod_s,
                        "texp_per_s": exp_prod, "frac_exp_peak": exp_prod / PEAK_EXP_TS,
                        "contraction_tflops": flops / avg_prod_s / 1e12,
                        "hbm_bytes_per_launch": recorded_traffic("product")},
            "rowsum": {"launches": row_n, "avg_ms": avg_row_s * 1e3,
                       "texp_per_s": exp_row, "frac_exp_peak": exp_row / PEAK_EXP_TS,
                       "hbm_bytes_per_launch": recorded_traffic("rowsum")},
        },
    }
    del ws_p, ws_d, Y, V
    if args.calibration_copy > 0:
        src = torch.ones(args.calibration_copy << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        rec["calibration_copy_bytes"] = 2 * src.numel() * 4
        del src, dst
    if not args.no_top64:
        top = lanczos_top64_leg(fd, torch, wl, X)
        rec["lanczos_top64_s"] = top["seconds"]
        rec["lanczos_top64"] = top
    if not args.no_torus6:
        log("flat 6-torus sweep")
        rec["torus6_sweep"] = torus6_sweep_leg(fd, torch, dev, 10)
    del X
    torch.cuda.empty_cache()
    if args.lanczos:
        rec["lanczos"] = lanczos_leg(fd, torch, dev)
    if args.continuation:
        rec["continuation"] = continuation_leg(fd, torch, dev, cold=args.continuation_cold)
    if args.stress:
        rec["stress"] = stress_leg(fd, torch, dev, args.stress_iters)
    if args.paper_t6:
        rec["paper_t6"] = paper_t6_leg(fd, torch, dev)
    if args.paper_t6_flow:
        rec["paper_t6_flow"] = paper_t6_flow_leg(fd, torch, dev, args.paper_t6_flow)
    if not args.no_cpu_baseline:
        log("CPU oracle baseline")
        rec["cpu_baseline"] = cpu_baseline(wl.X, beta, b, args.cpu_seconds,
                                           "molecule-like N=2^20 D=30")
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
