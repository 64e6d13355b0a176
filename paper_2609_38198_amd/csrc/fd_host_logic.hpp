// Host-side decision logic of the eigensolver, the continuation and the beta
// flow, free of HIP: the library drives it with device probes, and a CPU test
// program (built with the address and undefined-behaviour sanitizers) drives
// it with mocked probes.  Nothing here touches device memory.
#pragma once

#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <string>
#include <vector>

#include "flashdiff.h"

namespace fd {
namespace logic {

inline int64_t up_to(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------- eigensolver

constexpr double KAPPA_P = 10.0;   // safety factor of the Perron wall (eq. perronwall)
constexpr double ETA_FP32 = 1e-7;  // precision scale of float32 kernel data
constexpr double ETA_BF16 = 8e-3;  // precision scale of bfloat16 kernel data

// eta of the data type the kernel is evaluated from (footnote to eq. perronwall)
inline double eta_of(fd_dtype xt) { return xt == FD_BF16 ? ETA_BF16 : ETA_FP32; }

struct SolverLayout {
  int b = 0, k = 0, keep = 0, kk = 0, mm = 0;
  int m_first = 0;  // basis width of the first restart cycle
  bool dense = false;
};

// Basis capacity.  The first restart cycle has m_first = kk rounded up to
// whole blocks, plus as many again (at least two blocks): well-separated
// spectra converge in a few such cycles.  The capacity (four times that, at
// most 1024 columns) is what later cycles may grow to: on clustered spectra
// (the top k within 1e-3 of 1, gaps near the tolerance) thick restart
// converges only when each cycle adds many blocks.  Returns an empty string,
// or why the options are unusable.
// Default number of Ritz vectors kept beyond k: k itself (at least b), as
// far as k + keep + b fits the capacity.  A buffer as deep as the wanted set
// lets the pairs at the cluster edge converge with the rest: measured against
// keep = b, the molecule-like top 64 (N = 2^20, b = 32) takes 8 block products
// instead of 9, the 2-torus top 16 (b = 8) 32 instead of 57, the noisy
// 6-torus ladder 2,004 instead of 2,367.
inline int default_keep(int b, int k, int limit) {
  return std::max(b, std::min(k, limit - k - b));
}

inline std::string solver_layout(int64_t N, int b, int k, int keep_opt, int max_basis_blocks,
                                 SolverLayout& L) {
  L = SolverLayout{};
  L.b = b;
  L.k = k;
  const int cap = (1024 / b) * b;  // projected eigensolve limit
  L.keep = keep_opt >= 0 ? keep_opt
                         : default_keep(b, k, max_basis_blocks > 0 ? max_basis_blocks * b : cap);
  L.kk = k + L.keep;
  const int first = int(up_to(L.kk, b) + std::max<int64_t>(2 * b, up_to(L.kk, b)));
  int mm = max_basis_blocks > 0 ? max_basis_blocks * b : 4 * first;
  mm = std::min(mm, cap);
  if (N <= mm) {
    L.dense = true;
    L.mm = int(N);
    L.kk = int(N);
    L.m_first = int(N);
    return "";
  }
  L.mm = mm;
  L.m_first = std::min(first, mm);
  if (L.kk + b > mm)
    return "basis too small: need k + keep + b <= max_basis_blocks * b (and <= 1024)";
  return "";
}

// Basis width of the next restart cycle: doubled (up to the capacity) when
// the cycle just finished made little progress, i.e. converged fewer new
// leading pairs than b or half of those still missing, whichever is smaller;
// kept otherwise.  Every cycle ends in a thick restart whose new block holds
// the residuals of the leading unconverged pairs and random vectors:
// directions a Krylov space of one start block cannot reach (an eigenspace of
// multiplicity above b) keep entering the basis.
inline int next_cycle_width(const SolverLayout& L, int width, int nconv_before, int nconv) {
  // a cycle narrower than the first width (the one-block check after a warm
  // start) is followed by a cycle of the first width: further one-block
  // cycles would each end in a restart that drops most of their Krylov space
  if (width < L.m_first) return L.m_first;
  const int need = std::min(L.b, std::max(1, (L.k - nconv_before) / 2));
  if (nconv - nconv_before >= need) return width;
  return std::min(L.mm, 2 * width);
}

// Width of the first cycle after the Rayleigh-Ritz of a warm start (nkeep
// Ritz pairs kept): one block, so that a start already close to the answer is
// checked after a single product; later cycles grow by next_cycle_width.
inline int warm_cycle_width(const SolverLayout& L, int nkeep) {
  return std::min(L.m_first, nkeep + L.b);
}

// Leading Ritz pairs whose residual is at most tol.
inline int count_converged(const double* res, int k, double tol) {
  int n = 0;
  while (n < k && res[n] <= tol) ++n;
  return n;
}

// Columns whose residuals span the next block at a restart: the leading
// unconverged Ritz pairs among the nkeep kept, at most b of them.
inline int restart_columns(const double* res, int nkeep, int b, double tol, int* sel) {
  int ns = 0;
  for (int c = 0; c < nkeep && ns < b; ++c)
    if (res[c] > tol) sel[ns++] = c;
  return ns;
}

// Perron gap of Ritz values (theta descending).
inline double perron_gap(double th0, double th1) {
  return th0 != 0.0 ? (th0 - th1) / std::fabs(th0) : 0.0;
}

// Perron wall (eq. perronwall): once the Perron pair has converged, its Ritz
// gap bounds the true gap from above (theta_1 <= lambda_1); at or below
// kappa_P eta the leading eigenspace cannot be resolved from data of this
// precision, and further restarts cannot change that.
inline bool at_perron_wall(int m, double th0, double th1, double res0, double tol, double eta) {
  return m >= 2 && res0 <= tol && perron_gap(th0, th1) <= KAPPA_P * eta;
}

// ---------------------------------------------------------------- continuation

// Step whose Markov vectors start step t when the prefix grows: the last step
// solved at the previous prefix with the same beta if there is one, else the
// previous step (`last`).  level_beta / level_slot list the steps of the
// previous prefix in order.
inline int64_t nystrom_source(const std::vector<float>& level_beta,
                              const std::vector<int64_t>& level_slot, float beta_t,
                              int64_t last) {
  int64_t src = last;
  for (size_t e = 0; e < level_beta.size() && e < level_slot.size(); ++e)
    if (level_beta[e] == beta_t) src = level_slot[e];
  return src;
}

// ---------------------------------------------------------------- beta flow
//
// Sec. 2.3 ("beta-function flow"): dyadic probes from beta_0, the empirical
// potential V = V_bias + V_stat + V_mach over log beta, the bracketing rule
// with a quadratic vertex probe, and the Perron wall.

struct FlowParams {
  double eta, kappa, p;
};

struct FlowProbe {
  double beta = 0.0, s_off = 0.0, gap = 0.0, v_bias = 0.0, v_mach = 0.0;
  double n_eff = NAN, v_stat = NAN, v_total = NAN, d_hat = NAN, seconds = 0.0;
  bool admissible = false, converged = false;
  int role = 0, matvecs = 0, nconv = 0;
  std::vector<double> evals;
  bool complete() const { return !std::isnan(v_total); }
};

// Quantities a probe knows on its own, from its k eigenvalues (Perron first):
// g_P, V_bias = median_j -log(lambda_j / lambda_0) over the nontrivial pairs
// (eq. vbias), V_mach = (kappa_P eta / g_P)^p (eq. vmach) and the
// admissibility g_P > kappa_P eta (eq. perronwall).
inline void probe_stats(FlowProbe& pr, int k, const FlowParams& fp) {
  pr.evals.resize(size_t(std::max(k, 2)), 0.0);
  const double l0 = pr.evals[0];
  pr.gap = perron_gap(l0, pr.evals[1]);
  std::vector<double> h;
  for (int j = 1; j < k; ++j) h.push_back(-std::log(pr.evals[size_t(j)] / l0));
  std::sort(h.begin(), h.end());
  const size_t n = h.size();
  pr.v_bias = n == 0 ? 0.0 : (n % 2 == 1) ? h[n / 2] : 0.5 * (h[n / 2 - 1] + h[n / 2]);
  pr.v_mach = pr.gap > 0.0 ? std::pow(fp.kappa * fp.eta / pr.gap, fp.p) : INFINITY;
  pr.admissible = pr.gap > fp.kappa * fp.eta;
}

// Quantities of `a` that need S_off at twice its bandwidth (probe c): n_eff
// (eq. neff), V_stat (eq. vstat), V (eq. vtotal) and d_hat (eq. dhat).
inline void flow_complete(FlowProbe& a, const FlowProbe& c, int64_t N) {
  a.n_eff = a.s_off * a.s_off / (double(N) * c.s_off);
  a.v_stat = 1.0 / std::sqrt(a.n_eff * a.v_bias);
  a.v_total = a.v_bias + a.v_stat + a.v_mach;
  a.d_hat = -2.0 * (std::log(c.s_off) - std::log(a.s_off)) / (std::log(c.beta) - std::log(a.beta));
}

// Three consecutive complete probes bracket a minimum of V with V_bias
// falling and V_stat or V_mach rising between the outer two.
inline bool flow_brackets(const FlowProbe& a, const FlowProbe& m, const FlowProbe& c) {
  return a.v_total > m.v_total && c.v_total > m.v_total && c.v_bias < a.v_bias &&
         (c.v_stat > a.v_stat || c.v_mach > a.v_mach);
}

// Vertex abscissa of the parabola through (x_i, y_i), clamped to [x0, x2].
inline double flow_vertex(const double x[3], const double y[3]) {
  const double den = (x[0] - x[1]) * (x[0] - x[2]) * (x[1] - x[2]);
  const double A = (x[2] * (y[1] - y[0]) + x[1] * (y[0] - y[2]) + x[0] * (y[2] - y[1])) / den;
  const double B =
      (x[2] * x[2] * (y[0] - y[1]) + x[1] * x[1] * (y[2] - y[0]) + x[0] * x[0] * (y[1] - y[2])) /
      den;
  const double v = -B / (2.0 * A);
  return std::min(std::max(v, x[0]), x[2]);
}

struct FlowOutcome {
  bool any = false;  // at least one admissible probe
  int reason = FD_FLOW_BUDGET;
  FlowProbe fin;     // the probe at the achieved bandwidth
};

// One sweep of the flow from `beta`: dyadic probes until a bracket (then one
// vertex probe), the wall, max_probes or a bandwidth outside the driver's
// exponent range (not probed; the sweep ends as on the probe budget).  The
// driver runs the probes and owns their vectors:
//   bool drv.in_range(double beta)   whether a probe at beta can be run;
//   FlowProbe drv.probe(double beta, int role, int t, bool from_keep)
//       solve at beta (role 0 dyadic, 1 vertex, 2 final re-solve), its Markov
//       vectors into the driver's "new" slot, started from the "keep" slot
//       when from_keep;
//   void drv.accept()   the latest probe is admissible: "new" becomes "keep";
//   void drv.record(const FlowProbe&, bool replace_last)   report a probe.
// On return with any == true the driver's latest solve is the one at fin.beta
// and its Markov vectors are in "keep".
template <class Driver>
FlowOutcome run_flow_logic(Driver& drv, int64_t N, double beta, bool warm, int max_probes) {
  FlowOutcome res;
  std::vector<FlowProbe> pr;  // admissible dyadic probes
  bool have_keep = warm;      // "keep" holds the latest admissible probe (or the warm start)
  double in_q = -1.0;         // bandwidth of the driver's latest solve
  int reason = FD_FLOW_BUDGET;
  FlowProbe fin;
  bool fin_in_q = false;
  for (int t = 0; t < max_probes; ++t) {
    if (!drv.in_range(beta)) {
      reason = FD_FLOW_RANGE;
      break;
    }
    FlowProbe p = drv.probe(beta, 0, t, have_keep);
    in_q = beta;
    if (!p.admissible) {
      drv.record(p, false);
      reason = FD_FLOW_WALL;
      break;
    }
    if (!pr.empty()) {
      flow_complete(pr.back(), p, N);
      drv.record(pr.back(), true);
    }
    pr.push_back(p);
    drv.record(p, false);
    drv.accept();
    have_keep = true;
    std::vector<size_t> done;
    for (size_t i = 0; i < pr.size(); ++i)
      if (pr[i].complete()) done.push_back(i);
    const size_t nd = done.size();
    if (nd >= 3 && flow_brackets(pr[done[nd - 3]], pr[done[nd - 2]], pr[done[nd - 1]])) {
      const FlowProbe& pa = pr[done[nd - 3]];
      const FlowProbe& pm = pr[done[nd - 2]];
      const FlowProbe& pc = pr[done[nd - 1]];
      const double xs[3] = {std::log(pa.beta), std::log(pm.beta), std::log(pc.beta)};
      const double ys[3] = {pa.v_total, pm.v_total, pc.v_total};
      const double bv = std::exp(flow_vertex(xs, ys));
      FlowProbe v = drv.probe(bv, 1, t, true);
      in_q = bv;
      drv.record(v, false);
      reason = FD_FLOW_BRACKET;
      if (v.admissible) {
        fin = v;
        fin_in_q = true;
      } else {
        fin = pm;
      }
      break;
    }
    beta *= 2.0;
  }
  res.reason = reason;
  if (pr.empty()) return res;
  res.any = true;
  if (reason != FD_FLOW_BRACKET) {
    fin = pr.back();
    if (reason == FD_FLOW_BUDGET || reason == FD_FLOW_RANGE) {
      for (const FlowProbe& q : pr)
        if (q.complete() && (!fin.complete() || q.v_total < fin.v_total)) fin = q;
    }
    fin_in_q = in_q == fin.beta;
  }
  if (!fin_in_q) {
    // the selected probe's vectors were overwritten: solve again from the
    // latest admissible probe's Markov vectors
    FlowProbe r = drv.probe(fin.beta, 2, max_probes, true);
    drv.record(r, false);
    fin.evals = r.evals;
    fin.converged = r.converged;
    fin.nconv = r.nconv;
    drv.accept();
  } else if (fin.role == 0) {
    // the latest dyadic probe: its Markov vectors were accepted already
  } else {
    drv.accept();
  }
  res.fin = fin;
  return res;
}

}  // namespace logic
}  // namespace fd
