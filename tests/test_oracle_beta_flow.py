"""Pins of the oracle's beta-function flow (Sec. 2.3) against facts that do
not depend on its own formulas: closed-form initial bandwidths, exact
spectra, the paper's statement that n_eff equals k for k equally weighted
interactions per row, the intrinsic dimension of flat grid tori (circulant
closed form), an exact parabola, and the sweep's three exits on mocked
probe sequences."""
import math

import numpy as np
import pytest

from oracle import beta_flow as bf
from oracle import normalise as on
from oracle import torus_grid as tg


def circle(N, R, dim=2):
    t = 2 * np.pi * np.arange(N) / N
    X = np.zeros((N, dim))
    X[:, 0] = R * np.cos(t)
    X[:, 1] = R * np.sin(t)
    return X + 5.0  # an offset the centring must remove


@pytest.mark.parametrize("R,want", [(3.0, 1.0 / 18.0), (1.0, 0.1), (2.0, 0.1)])
def test_beta0_closed_form(R, want):
    # centred points on a circle of radius R: mean ||x||^2 = R^2
    assert bf.beta0(circle(360, R)) == pytest.approx(want, rel=1e-12)


def test_v_bias_exact_spectrum():
    ev = np.exp(-np.array([0.0, 1.0, 2.0, 3.0, 7.0]))
    assert bf.v_bias(ev) == pytest.approx(2.5, rel=1e-12)  # median of 1, 2, 3, 7
    assert bf.v_bias(2.0 * ev) == pytest.approx(2.5, rel=1e-12)  # scale invariant


@pytest.mark.parametrize("k", [1, 3, 7])
def test_n_eff_counts_equal_interactions(k):
    # groups of k + 1 coincident points, groups far apart: every row has k
    # interactions of weight 1 at any beta, so n_eff = k (text after eq. neff)
    rng = np.random.default_rng(k)
    centres = rng.normal(size=(40, 3)) * 100.0
    X = np.repeat(centres, k + 1, axis=0)
    N = X.shape[0]
    s1 = on.normalise(X, 0.5, 0.5).s_off
    s2 = on.normalise(X, 1.0, 0.5).s_off
    assert s1 == pytest.approx(N * k, rel=1e-12)
    assert bf.n_eff(s1, s2, N) == pytest.approx(k, rel=1e-12)


def simplex_clusters(k, h, groups=40):
    """Groups of k + 1 points at the vertices of a regular simplex of edge h
    (scaled unit vectors of R^(k+1)), group centres 100 apart on a line."""
    centres = np.zeros((groups, k + 1))
    centres[:, 0] = 100.0 * np.arange(groups)
    verts = np.eye(k + 1) * (h / math.sqrt(2.0))
    return (centres[:, None, :] + verts[None, :, :]).reshape(-1, k + 1)


@pytest.mark.parametrize("k", [1, 3, 7])
def test_n_eff_orientation_on_equidistant_neighbours(k):
    # every row has k neighbours at squared distance h^2 and nothing else in
    # reach: S_off(beta) = N k exp(-beta h^2), S_off(2 beta) = N k
    # exp(-2 beta h^2), and n_eff = k at any beta (text after eq. neff).  The
    # arguments taken the other way round give k exp(-3 beta h^2).
    h2, beta = 2.0, 0.5
    X = simplex_clusters(k, math.sqrt(h2))
    N = X.shape[0]
    s1 = on.normalise(X, beta, 0.5).s_off
    s2 = on.normalise(X, 2 * beta, 0.5).s_off
    assert s1 == pytest.approx(N * k * math.exp(-beta * h2), rel=1e-10)
    assert s2 == pytest.approx(N * k * math.exp(-2 * beta * h2), rel=1e-10)
    assert bf.n_eff(s1, s2, N) == pytest.approx(k, rel=1e-10)
    assert abs(bf.n_eff(s2, s1, N) - k) > 0.5 * k


@pytest.mark.parametrize("counts", [(256, 256), (512, 256)])
def test_n_eff_heat_regime_closed_form(counts):
    # flat grid torus of unit circles in the heat regime (kernel much wider
    # than the grid spacing, much narrower than the circles): the row sums
    # are a Riemann sum of a Gaussian, q - 1 ~ rho (pi / beta)^(d/2) with
    # rho = N / (2 pi)^d, so n_eff ~ rho (2 pi / beta)^(d/2) = N beta^(-d/2)
    # (2 pi)^(-d/2).  The circulant closed form gives q exactly.  The
    # swapped orientation is 2^(3d/2) = 8 times smaller at d = 2.
    d, beta = 2, 20.0
    N = int(np.prod(counts))
    s1 = N * (tg.degree(counts, beta) - 1.0)
    s2 = N * (tg.degree(counts, 2 * beta) - 1.0)
    want = N / (2 * np.pi) ** d * (2 * np.pi / beta) ** (d / 2)
    assert bf.n_eff(s1, s2, N) == pytest.approx(want, rel=0.02)
    assert bf.n_eff(s2, s1, N) < want / 4


def test_v_stat_definition():
    assert bf.v_stat(25.0, 4.0) == pytest.approx(0.1, rel=1e-15)


@pytest.mark.parametrize("counts,d", [((256, 256), 2), ((64, 64, 64), 3)])
def test_d_hat_recovers_grid_dimension(counts, d):
    # flat grid torus, kernel wider than the spacing and narrower than the
    # circles: S_off ~ beta^(-d/2), so d_hat ~ d (eq. dhat)
    N = int(np.prod(counts))
    beta = 20.0 if d == 2 else 8.0
    s1 = N * (tg.degree(counts, beta) - 1.0)
    s2 = N * (tg.degree(counts, 2 * beta) - 1.0)
    assert bf.d_hat(s1, s2, beta, 2 * beta) == pytest.approx(d, rel=0.05)


def test_parabola_vertex_exact():
    x = [0.0, 0.5, 1.2]
    y = [3 * (v - 0.7) ** 2 + 1 for v in x]
    assert bf.parabola_vertex(x, y) == pytest.approx(0.7, rel=1e-12)


def _mock(vb, soff, gaps, beta0=0.1):
    """Probe callable from per-probe V_bias, S_off and Perron gaps (index by
    the dyadic step; the vertex probe reuses the nearest step's values)."""
    def probe(beta):
        i = int(round(math.log2(beta / beta0)))
        i = max(0, min(i, len(vb) - 1))
        # evals with lambda_0 = 1, lambda_1 = 1 - gap and median -log = vb
        ev = np.array([1.0, 1.0 - gaps[i], math.exp(-vb[i]), math.exp(-vb[i])])
        return bf.make_probe(beta, ev, soff[i])
    return probe


def test_flow_probes_carry_n_eff_of_equidistant_neighbours():
    # the flow's own bookkeeping (each probe completed by the next dyadic
    # probe) must give n_eff = k on every complete probe when S_off follows
    # the equidistant-neighbour law N k exp(-beta h^2) of the simplex set
    # (that set itself is disconnected, so its Perron gap is 0: the probes
    # take an admissible mocked spectrum and this S_off)
    k, h2, N = 3, 1.0, 120
    vb = [4.0, 2.0, 1.0, 0.5]
    soff = [N * k * math.exp(-0.1 * 2 ** i * h2) for i in range(4)]
    F = bf.flow(_mock(vb, soff, [0.5] * 4), N, 0.1, max_probes=4)
    done = [p for p in F.probes if p.n_eff is not None]
    assert len(done) == 3
    for p in done:
        assert p.n_eff == pytest.approx(k, rel=1e-12)


def test_flow_brackets_known_minimum():
    N = 1000
    vb = [4.0, 2.0, 1.0, 0.5, 0.25, 0.12, 0.06]
    # S_off halving per step until step 3, then falling faster: V_stat grows
    soff = [N * 400 / 2 ** i for i in range(4)] + [N * 400 / 2 ** 3 / 8 ** j for j in range(1, 4)]
    gaps = [0.5] * 7
    F = bf.flow(_mock(vb, soff, gaps), N, 0.1, max_probes=7)
    assert F.reason == "bracket"
    Vs = [p.v_total for p in F.probes if p.v_total is not None]
    m = int(np.argmin(Vs))
    assert F.bracket == m
    lo, hi = F.probes[m - 1].beta, F.probes[m + 1].beta
    assert lo <= F.beta_x <= hi


def test_flow_stops_at_the_wall():
    N = 1000
    vb = [4.0, 2.0, 1.0, 0.5, 0.25, 0.12]
    soff = [N * 400 / 2 ** i for i in range(6)]
    gaps = [0.5, 0.2, 1e-3, 2e-5, 1e-7, 1e-8]  # step 4 is past kappa * eta = 1e-6
    F = bf.flow(_mock(vb, soff, gaps), N, 0.1, max_probes=6)
    assert F.reason == "wall"
    assert len(F.probes) == 4
    assert F.beta_x == pytest.approx(0.1 * 2 ** 3)


def test_flow_budget_takes_smallest_complete_potential():
    N = 1000
    vb = [4.0, 2.0, 1.0, 0.5]
    soff = [N * 400 / 2 ** i for i in range(4)]
    F = bf.flow(_mock(vb, soff, [0.5] * 4), N, 0.1, max_probes=4)
    assert F.reason == "budget"
    done = [p for p in F.probes if p.v_total is not None]
    assert F.final is min(done, key=lambda p: p.v_total)


def test_flow_on_two_torus_heat_regime():
    # 2048 points of the flat 2-torus, alpha = 1/2, 16 pairs: V_bias ~ 1/beta
    # and d_hat -> 2 in the heat regime; the sweep brackets a minimum
    from paper_2609_38198_amd import inputs
    w = inputs.torus2()
    F = bf.flow(bf.dense_probe(w.X, 0.5, 16), w.N, bf.beta0(w.X), max_probes=12)
    assert F.reason == "bracket"
    heat = [p for p in F.probes if p.v_total is not None and p.beta >= 3.0]
    assert heat
    for p in heat:
        assert p.d_hat == pytest.approx(2.0, rel=0.1)
    for a, c in zip(heat, heat[1:]):
        assert a.v_bias / c.v_bias == pytest.approx(2.0, rel=0.15)


def test_cascade_chains_levels_from_the_previous_selection():
    # level 0 (bf16: kappa * eta = 0.08) stops at its wall; level 1 (fp32)
    # starts at level 0's achieved bandwidth and continues to a bracket
    N = 1000
    vb = [4.0, 2.0, 1.0, 0.5, 0.25, 0.12, 0.06]
    soff = [N * 400 / 2 ** i for i in range(4)] + [N * 400 / 2 ** 3 / 8 ** j for j in range(1, 4)]
    gaps = [0.5, 0.3, 0.05, 0.02, 0.01, 0.01, 0.01]

    def mock(dtype):
        def probe(beta):
            i = max(0, min(int(round(math.log2(beta / 0.1))), len(vb) - 1))
            ev = np.array([1.0, 1.0 - gaps[i], math.exp(-vb[i]), math.exp(-vb[i])])
            return bf.make_probe(beta, ev, soff[i], dtype)
        return probe

    flows = bf.cascade([mock("bf16"), mock("fp32")], N, 0.1, max_probes=7)
    lo, hi = flows
    assert lo.reason == "wall" and lo.beta_x == pytest.approx(0.2)
    assert hi.probes[0].beta == pytest.approx(lo.beta_x)
    alone = bf.flow(mock("fp32"), N, lo.beta_x, max_probes=7)
    assert hi.beta_x == pytest.approx(alone.beta_x) and hi.reason == alone.reason


def test_single_level_cascade_is_the_flow():
    from paper_2609_38198_amd import inputs
    w = inputs.torus2()
    probe = bf.dense_probe(w.X, 0.5, 8)
    (F,) = bf.cascade([probe], w.N, bf.beta0(w.X), max_probes=4)
    G = bf.flow(probe, w.N, bf.beta0(w.X), max_probes=4)
    assert F.beta_x == G.beta_x and F.reason == G.reason
    assert [p.beta for p in F.probes] == [p.beta for p in G.probes]
