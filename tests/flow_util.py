"""Probe-by-probe comparison of the library's beta flow with the oracle's."""
import numpy as np
import pytest


def dyadic(flow):
    return [p for p in flow.probes if p["role"] == 0 and p["admissible"]]


def v_mach_tol(r, gap_tol, p=6.0):
    # V_mach = (kappa_P eta / g)^p (eq. perronwall): the change it can take while
    # the gap moves within its parity interval [g - gap_tol, g + gap_tol]; no
    # bound once that interval reaches 0 (next to the wall the gap is resolved
    # only to the eigenvalue floor, reading 6)
    lo = r.gap - gap_tol
    if lo <= 0.0:
        return float("inf")
    return r.v_mach * ((r.gap / lo) ** p - 1.0)


def compare_probes(gpu, ref):
    # tolerances propagated from the parity bars of the inputs: eigenvalues to
    # max(1e-5 |lambda|, 1e-6) (so -log(lambda_j / lambda_0) to about 1e-5 absolute
    # and the gap to 1e-6 absolute), S_off to 1e-5 relative (n_eff to 1e-4)
    assert len(gpu) == len(ref.probes)
    for i, (g, r) in enumerate(zip(gpu, ref.probes)):
        msg = (f"probe {i}: beta {r.beta:.6g}; gpu s_off {g['s_off']:.8g} gap {g['gap_perron']:.6g} "
               f"v_bias {g['v_bias']:.6g} v_mach {g['v_mach']:.6g}; oracle s_off {r.s_off:.8g} "
               f"gap {r.gap:.6g} v_bias {r.v_bias:.6g} v_mach {r.v_mach:.6g}")
        assert g["beta"] == pytest.approx(r.beta, rel=1e-12), msg
        assert g["s_off"] == pytest.approx(r.s_off, rel=1e-5), msg
        gap_tol = max(1e-4 * r.gap, 1e-6)
        assert abs(g["gap_perron"] - r.gap) <= gap_tol, msg
        vb_tol = max(1e-4 * r.v_bias, 1e-5)
        assert abs(g["v_bias"] - r.v_bias) <= vb_tol, msg
        vm_tol = v_mach_tol(r, gap_tol)
        assert abs(g["v_mach"] - r.v_mach) <= vm_tol + 1e-300, msg
        if r.v_total is None:
            assert np.isnan(g["v_total"]), msg
            continue
        assert g["n_eff"] == pytest.approx(r.n_eff, rel=1e-4), msg
        vs_tol = r.v_stat * 0.5 * (1e-4 + vb_tol / r.v_bias)
        assert abs(g["v_stat"] - r.v_stat) <= vs_tol, msg
        assert abs(g["v_total"] - r.v_total) <= vb_tol + vs_tol + vm_tol, msg
        assert g["d_hat"] == pytest.approx(r.d_hat, abs=1e-3), msg
