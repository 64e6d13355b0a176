"""Bandwidth selection by the beta-function flow, float64 (test infrastructure).

Sec. 2.3 ("beta-function flow"), in the paper's order:

* initial bandwidth from the centred data, eq. beta0:
  beta_0 = min(0.1, 1 / (2 N^-1 sum_i ||x_i - mean||^2));
* dyadic probes beta -> 2 beta; each probe gives the Perron pair and the
  requested nontrivial pairs of M, and S_off(beta) = sum_{i != j} K_ij
  (= sum(q) - N, eq. before neff);
* spectral heat action V_bias = median_j(-log(lambda_j / lambda_0)) over the
  nontrivial modes (eq. vbias);
* effective sample size n_eff(beta) = S_off(beta)^2 / (N S_off(2 beta))
  (eq. neff), known once the next dyadic probe has run, and
  V_stat = 1 / sqrt(n_eff V_bias) (eq. vstat);
* machine-precision barrier V_mach = (kappa_P eta / g_P)^p and the hard
  admissibility g_P > kappa_P eta (eqs. vmach, perronwall);
* V = V_bias + V_stat + V_mach (eq. vtotal); a minimum is accepted when three
  consecutive probes bracket it with V_bias falling and V_stat or V_mach
  rising; a quadratic fit in log beta over the triplet gives the vertex,
  resolved by a final probe; if the Perron wall comes first, the last safe
  probe is the achieved bandwidth;
* intrinsic-dimension diagnostic d_hat = -2 dlog S_off / dlog beta over a
  dyadic pair (eq. dhat).
* precision cascade (last paragraph of Sec. 2.3): with several data types,
  one sweep per type, lowest precision first; each later sweep starts at the
  bandwidth the previous one selected, and the last sweep's selection is
  the result.

Readings where the text leaves a choice:
* ``k`` counts the Perron pair (k - 1 nontrivial modes enter V_bias);
* "V_bias falling and V_stat or V_mach rising" is compared between the two
  ends of the bracketing triplet;
* when the probe budget runs out first, the achieved bandwidth is the
  complete probe (V known) with the smallest V, else the last safe probe;
* a vertex probe that lands past the wall falls back to the bracket's middle.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Callable, List, Optional

import numpy as np

from . import diagnostics as od
from .eig import spectrum


def beta0(X: np.ndarray) -> float:
    """Initial bandwidth from the centred data (eq. beta0)."""
    Xd = np.asarray(X, dtype=np.float64)
    Xc = Xd - Xd.mean(axis=0)
    ms = float(np.mean(np.sum(Xc * Xc, axis=1)))
    return min(0.1, 1.0 / (2.0 * ms))


def v_bias(evals) -> float:
    """Median of -log(lambda_j / lambda_0) over the nontrivial modes (eq. vbias)."""
    ev = np.asarray(evals, dtype=np.float64)
    return float(np.median(-np.log(ev[1:] / ev[0])))


def n_eff(s_off_beta: float, s_off_2beta: float, N: int) -> float:
    """Effective interaction count per row (eq. neff)."""
    return float(s_off_beta ** 2 / (N * s_off_2beta))


def v_stat(neff: float, vbias: float) -> float:
    """Relative statistical uncertainty (eq. vstat)."""
    return float(1.0 / math.sqrt(neff * vbias))


def d_hat(s_off_1: float, s_off_2: float, beta_1: float, beta_2: float) -> float:
    """Empirical intrinsic dimension from a pair of probes (eq. dhat)."""
    return float(-2.0 * (math.log(s_off_2) - math.log(s_off_1)) /
                 (math.log(beta_2) - math.log(beta_1)))


def parabola_vertex(x, y) -> float:
    """Abscissa of the vertex of the parabola through three points."""
    (x0, x1, x2), (y0, y1, y2) = x, y
    den = (x0 - x1) * (x0 - x2) * (x1 - x2)
    a = (x2 * (y1 - y0) + x1 * (y0 - y2) + x0 * (y2 - y1)) / den
    b = (x2 * x2 * (y0 - y1) + x1 * x1 * (y2 - y0) + x0 * x0 * (y1 - y2)) / den
    return float(-b / (2.0 * a))


@dataclass
class Probe:
    beta: float
    evals: np.ndarray
    s_off: float
    gap: float
    admissible: bool
    v_bias: float
    v_mach: float
    n_eff: Optional[float] = None
    v_stat: Optional[float] = None
    v_total: Optional[float] = None
    d_hat: Optional[float] = None


@dataclass
class Flow:
    probes: List[Probe] = field(default_factory=list)
    beta_x: float = float("nan")       # achieved bandwidth
    reason: str = ""                   # "bracket", "wall" or "budget"
    bracket: Optional[int] = None      # index of the bracket's middle probe
    final: Optional[Probe] = None      # probe at beta_x


def make_probe(beta: float, evals, s_off: float, dtype: str = "fp32") -> Probe:
    ev = np.asarray(evals, dtype=np.float64)
    g = od.perron_gap(ev)
    return Probe(beta=beta, evals=ev, s_off=float(s_off), gap=g,
                 admissible=od.wall_admissible(g, dtype), v_bias=v_bias(ev),
                 v_mach=od.v_mach(g, dtype) if g > 0 else float("inf"))


def dense_probe(X: np.ndarray, alpha: float, k: int, dtype: str = "fp32"):
    """Probe callable: dense float64 spectrum of M and S_off at beta."""
    def probe(beta: float) -> Probe:
        sp = spectrum(X, beta, alpha, k)
        return make_probe(beta, sp.evals, sp.norm.s_off, dtype)
    return probe


def _complete(prev: Probe, nxt: Probe, N: int) -> None:
    """Fill the quantities of `prev` that need S_off at twice its beta."""
    prev.n_eff = n_eff(prev.s_off, nxt.s_off, N)
    prev.v_stat = v_stat(prev.n_eff, prev.v_bias)
    prev.v_total = prev.v_bias + prev.v_stat + prev.v_mach
    prev.d_hat = d_hat(prev.s_off, nxt.s_off, prev.beta, nxt.beta)


def _brackets(a: Probe, m: Probe, c: Probe) -> bool:
    return (a.v_total > m.v_total < c.v_total and c.v_bias < a.v_bias
            and (c.v_stat > a.v_stat or c.v_mach > a.v_mach))


def flow(probe: Callable[[float], Probe], N: int, beta_start: float,
         max_probes: int = 24) -> Flow:
    """Dyadic sweep from beta_start until a bracket, the wall or the budget."""
    F = Flow()
    beta = beta_start
    while len(F.probes) < max_probes:
        p = probe(beta)
        if not p.admissible:
            F.reason = "wall"
            break
        if F.probes:
            _complete(F.probes[-1], p, N)
        F.probes.append(p)
        done = [q for q in F.probes if q.v_total is not None]
        if len(done) >= 3 and _brackets(done[-3], done[-2], done[-1]):
            a, m, c = done[-3], done[-2], done[-1]
            F.bracket = len(done) - 2
            x = [math.log(q.beta) for q in (a, m, c)]
            xv = min(max(parabola_vertex(x, [q.v_total for q in (a, m, c)]), x[0]), x[2])
            fin = probe(math.exp(xv))
            if fin.admissible:
                F.final = fin
            else:
                F.final = m
            F.beta_x = F.final.beta
            F.reason = "bracket"
            return F
        beta *= 2.0
    if not F.reason:
        F.reason = "budget"
    done = [q for q in F.probes if q.v_total is not None]
    if F.reason == "budget" and done:
        F.final = min(done, key=lambda q: q.v_total)
    elif F.probes:
        F.final = F.probes[-1]
    F.beta_x = F.final.beta if F.final is not None else float("nan")
    return F


def cascade(levels: List[Callable[[float], Probe]], N: int, beta_start: float,
            max_probes: int = 24) -> List[Flow]:
    """Precision cascade: one flow per probe callable (one data type each,
    lowest precision first), each from the previous flow's achieved
    bandwidth.  Returns the flows run; the last one holds the result."""
    flows: List[Flow] = []
    beta = beta_start
    for probe in levels:
        F = flow(probe, N, beta, max_probes)
        flows.append(F)
        if not F.probes:
            break
        beta = F.beta_x
    return flows
