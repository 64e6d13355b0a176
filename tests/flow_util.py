"""Probe-by-probe comparison of the library's beta flow with the oracle's."""
import numpy as np
import pytest


def dyadic(flow):
    return [p for p in flow.probes if p["role"] == 0 and p["admissible"]]


def compare_probes(gpu, ref):
    # tolerances propagated from the parity bars of the inputs: eigenvalues to
    # max(1e-5 |lambda|, 1e-6) (so -log(lambda_j / lambda_0) to about 1e-5 absolute
    # and the gap to 1e-6 absolute), S_off to 1e-5 relative (n_eff to 1e-4)
    assert len(gpu) == len(ref.probes)
    for g, r in zip(gpu, ref.probes):
        assert g["beta"] == pytest.approx(r.beta, rel=1e-12)
        assert g["s_off"] == pytest.approx(r.s_off, rel=1e-5)
        gap_tol = max(1e-4 * r.gap, 1e-6)
        assert abs(g["gap_perron"] - r.gap) <= gap_tol
        vb_tol = max(1e-4 * r.v_bias, 1e-5)
        assert abs(g["v_bias"] - r.v_bias) <= vb_tol
        vm_tol = r.v_mach * 6.0 * gap_tol / r.gap
        assert abs(g["v_mach"] - r.v_mach) <= vm_tol + 1e-300
        if r.v_total is None:
            assert np.isnan(g["v_total"])
            continue
        assert g["n_eff"] == pytest.approx(r.n_eff, rel=1e-4)
        vs_tol = r.v_stat * 0.5 * (1e-4 + vb_tol / r.v_bias)
        assert abs(g["v_stat"] - r.v_stat) <= vs_tol
        assert abs(g["v_total"] - r.v_total) <= vb_tol + vs_tol + vm_tol
        assert g["d_hat"] == pytest.approx(r.d_hat, abs=1e-3)
