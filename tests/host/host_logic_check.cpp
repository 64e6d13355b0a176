// CPU driver of the library's host-side decision logic (fd_host_logic.hpp),
// built with the address and undefined-behaviour sanitizers by
// tests/test_host_logic.py.  Two modes:
//   host_logic_check units        built-in checks of the eigensolver's and the
//                                 continuation's bookkeeping (exit status 0/1)
//   host_logic_check flow < spec  the beta-flow sweep over mocked probes read
//                                 from stdin; prints every record and the
//                                 outcome for comparison with the oracle's flow
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "fd_host_logic.hpp"

using namespace fd::logic;

static int failures = 0;
#define CHECK(cond)                                                      \
  do {                                                                   \
    if (!(cond)) {                                                       \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                        \
    }                                                                    \
  } while (0)

static int units() {
  SolverLayout L;
  // k = 64, b = 32, default keep (k): first cycle 256, capacity 1024
  CHECK(solver_layout(262144, 32, 64, -1, 0, L).empty());
  CHECK(!L.dense && L.kk == 128 && L.m_first == 256 && L.mm == 1024);
  // k = 16, b = 8: first cycle 64, capacity 256
  CHECK(solver_layout(2048, 8, 16, -1, 0, L).empty());
  CHECK(L.m_first == 64 && L.mm == 256);
  // the capacity never passes 1024 columns
  CHECK(solver_layout(1 << 21, 64, 64, 64, 0, L).empty());
  CHECK(L.mm == 1024 && L.m_first == 256);
  // an explicit capacity is honoured, and the first check never lies beyond it
  CHECK(solver_layout(1 << 20, 32, 64, -1, 6, L).empty());
  CHECK(L.mm == 192 && L.m_first == 192);
  // problems no larger than the capacity are solved in the full space
  CHECK(solver_layout(500, 32, 64, -1, 0, L).empty());
  CHECK(L.dense && L.mm == 500 && L.kk == 500);
  // a basis too small for k + keep + b is refused
  CHECK(!solver_layout(1 << 20, 32, 64, -1, 3, L).empty());

  // default keep: k (at least b) as far as k + keep + b fits the capacity
  CHECK(default_keep(32, 64, 1024) == 64 && default_keep(8, 4, 1024) == 8);
  CHECK(default_keep(32, 500, 1024) == 492 && default_keep(32, 64, 192) == 64);
  CHECK(default_keep(32, 64, 160) == 64 && default_keep(32, 64, 128) == 32);
  // restart cycles: the width doubles (up to the capacity) after a cycle that
  // converged fewer new leading pairs than min(b, half of those missing)
  CHECK(solver_layout(1 << 20, 32, 64, -1, 0, L).empty());
  CHECK(L.keep == 64 && L.kk == 128 && L.m_first == 256 && L.mm == 1024);
  CHECK(next_cycle_width(L, 256, 0, 59) == 256);
  CHECK(next_cycle_width(L, 256, 0, 31) == 512);
  CHECK(next_cycle_width(L, 512, 31, 40) == 1024);
  CHECK(next_cycle_width(L, 1024, 40, 41) == 1024);
  CHECK(next_cycle_width(L, 256, 10, 42) == 256);
  CHECK(next_cycle_width(L, 256, 56, 60) == 256);   // 4 of the 8 missing
  CHECK(next_cycle_width(L, 256, 56, 59) == 512);
  CHECK(solver_layout(1 << 20, 32, 64, -1, 8, L).empty());  // explicit capacity 256
  CHECK(L.keep == 64 && L.m_first == 256 && next_cycle_width(L, 256, 0, 0) == 256);
  CHECK(solver_layout(1 << 20, 32, 64, 32, 0, L).empty());  // explicit keep = b
  CHECK(L.kk == 96 && L.m_first == 192 && L.mm == 768);
  CHECK(solver_layout(4096, 8, 8, -1, 0, L).empty());  // k = 8, b = 8
  CHECK(L.m_first == 32 && next_cycle_width(L, 32, 3, 7) == 32);
  // after a warm start the first cycle is one block
  CHECK(warm_cycle_width(L, 8) == 16);
  CHECK(solver_layout(262144, 32, 64, -1, 0, L).empty());
  CHECK(warm_cycle_width(L, 64) == 96 && warm_cycle_width(L, 128) == 160);
  // after the one-block check the cycles take the first width, progress or not
  CHECK(next_cycle_width(L, 96, 0, 64) == 256 && next_cycle_width(L, 96, 0, 0) == 256);

  // convergence count stops at the first unconverged pair
  const double res[6] = {1e-7, 2e-6, 5e-5, 1e-8, 1e-9, 3e-4};
  CHECK(count_converged(res, 6, 1e-5) == 2);
  CHECK(count_converged(res, 1, 1e-5) == 1);
  CHECK(count_converged(res, 6, 1e-3) == 6);
  // restart block: the leading unconverged pairs, at most b of them
  int sel[4] = {-1, -1, -1, -1};
  CHECK(restart_columns(res, 6, 4, 1e-5, sel) == 2 && sel[0] == 2 && sel[1] == 5);
  CHECK(restart_columns(res, 6, 1, 1e-5, sel) == 1 && sel[0] == 2);
  CHECK(restart_columns(res, 2, 4, 1e-5, sel) == 0);

  // Perron wall: only once the Perron pair has converged, at gap <= kappa eta
  CHECK(at_perron_wall(64, 1.0, 1.0 - 5e-7, 1e-6, 1e-5, ETA_FP32));
  CHECK(!at_perron_wall(64, 1.0, 1.0 - 5e-7, 2e-5, 1e-5, ETA_FP32));
  CHECK(!at_perron_wall(64, 1.0, 1.0 - 2e-6, 1e-6, 1e-5, ETA_FP32));
  CHECK(at_perron_wall(64, 1.0, 0.95, 1e-6, 1e-5, ETA_BF16));
  CHECK(!at_perron_wall(1, 1.0, 0.0, 1e-6, 1e-5, ETA_FP32));
  CHECK(std::fabs(perron_gap(2.0, 1.5) - 0.25) < 1e-15);

  // continuation: the Nystrom source is the previous prefix's step with the
  // same beta, else the previous step
  const std::vector<float> lb = {0.5f, 1.f, 2.f, 4.f, 8.f};
  const std::vector<int64_t> ls = {0, 1, 2, 3, 4};
  CHECK(nystrom_source(lb, ls, 0.5f, 4) == 0);
  CHECK(nystrom_source(lb, ls, 4.f, 4) == 3);
  CHECK(nystrom_source(lb, ls, 16.f, 4) == 4);
  CHECK(nystrom_source({}, {}, 0.5f, 7) == 7);
  const std::vector<float> dup = {2.f, 2.f};
  const std::vector<int64_t> dups = {5, 6};
  CHECK(nystrom_source(dup, dups, 2.f, 6) == 6);

  // flow pieces: vertex of an exact parabola; probe statistics
  const double xs[3] = {0.0, 0.5, 1.2};
  double ys[3];
  for (int i = 0; i < 3; ++i) ys[i] = 3 * (xs[i] - 0.7) * (xs[i] - 0.7) + 1;
  CHECK(std::fabs(flow_vertex(xs, ys) - 0.7) < 1e-12);
  FlowProbe pr;
  pr.evals = {1.0, std::exp(-1.0), std::exp(-2.0), std::exp(-3.0), std::exp(-7.0)};
  probe_stats(pr, 5, FlowParams{1e-7, 10.0, 6.0});
  CHECK(std::fabs(pr.v_bias - 2.5) < 1e-12 && pr.admissible);
  CHECK(std::fabs(pr.gap - (1.0 - std::exp(-1.0))) < 1e-15);
  std::printf("units: %d failures\n", failures);
  return failures == 0 ? 0 : 1;
}

// Mocked probes: dyadic index i = round(log2(beta / beta0)) clamped to the
// table; eigenvalues {1, 1 - gap_i, exp(-vb_i), exp(-vb_i), ...} (k of them),
// S_off = soff_i.
struct MockDriver {
  double beta0;
  int k;
  FlowParams fp;
  std::vector<double> vb, soff, gap;
  int accepts = 0;
  double beta_max = INFINITY;  // exponent range of the mock
  bool in_range(double beta) const { return beta <= beta_max; }
  FlowProbe probe(double beta, int role, int t, bool from_keep) {
    (void)t;
    (void)from_keep;
    const int n = int(vb.size());
    int i = int(std::lround(std::log2(beta / beta0)));
    i = std::max(0, std::min(i, n - 1));
    FlowProbe p;
    p.beta = beta;
    p.role = role;
    p.s_off = soff[size_t(i)];
    p.evals.assign(size_t(k), std::exp(-vb[size_t(i)]));
    p.evals[0] = 1.0;
    p.evals[1] = 1.0 - gap[size_t(i)];
    p.converged = true;
    probe_stats(p, k, fp);
    return p;
  }
  void accept() { ++accepts; }
  void record(const FlowProbe& p, bool replace_last) {
    std::printf("record %d %d %.17g %.17g %.17g %.17g %.17g %.17g %.17g %.17g %.17g %d\n",
                replace_last ? 1 : 0, p.role, p.beta, p.s_off, p.gap, p.v_bias, p.v_mach,
                p.n_eff, p.v_stat, p.v_total, p.d_hat, p.admissible ? 1 : 0);
  }
};

// The sweep stops before a bandwidth outside the exponent range and chooses
// as on the probe budget: V_bias falls and S_off does not, so no bracket; the
// probe at 8 beta0 would be out of range
static int flow_range_units() {
  int fails = 0;
  const std::vector<double> vb = {4.0, 3.0, 2.2, 1.6, 1.2, 0.9}, so = {1, 1, 1, 1, 1, 1},
                            gap = {0.5, 0.4, 0.3, 0.2, 0.1, 0.05};
  MockDriver drv{1.0, 8, FlowParams{1e-7, 10.0, 6.0}, vb, so, gap, 0, 5.0};
  const FlowOutcome R = run_flow_logic(drv, 1000, 1.0, false, 6);
  if (!(R.any && R.reason == FD_FLOW_RANGE && R.fin.beta <= 4.0 && drv.accepts >= 3)) ++fails;
  MockDriver first{1.0, 8, FlowParams{1e-7, 10.0, 6.0}, vb, so, gap, 0, 0.5};
  const FlowOutcome R0 = run_flow_logic(first, 1000, 1.0, false, 6);
  if (!(!R0.any && R0.reason == FD_FLOW_RANGE && first.accepts == 0)) ++fails;
  std::fprintf(stderr, "flow range units: %d failures\n", fails);
  return fails;
}

static int flow() {
  long long N = 0;
  int max_probes = 0, k = 0, warm = 0, n = 0;
  double beta0 = 0, eta = 0, kappa = 0, p = 0;
  if (std::scanf("%lld %lf %d %lf %lf %lf %d %d %d", &N, &beta0, &max_probes, &eta, &kappa, &p,
                 &k, &warm, &n) != 9 || n < 1 || n > 1000 || k < 2 || k > 1000) {
    std::fprintf(stderr, "bad spec\n");
    return 2;
  }
  MockDriver drv{beta0, k, FlowParams{eta, kappa, p}, {}, {}, {}, 0, INFINITY};
  for (int i = 0; i < n; ++i) {
    double a, b, c;
    if (std::scanf("%lf %lf %lf", &a, &b, &c) != 3) {
      std::fprintf(stderr, "bad row %d\n", i);
      return 2;
    }
    drv.vb.push_back(a);
    drv.soff.push_back(b);
    drv.gap.push_back(c);
  }
  const FlowOutcome R = run_flow_logic(drv, N, beta0, warm != 0, max_probes);
  std::printf("outcome %d %d %.17g %d\n", R.any ? 1 : 0, R.reason, R.any ? R.fin.beta : NAN,
              drv.accepts);
  return 0;
}

int main(int argc, char** argv) {
  if (argc == 2 && std::strcmp(argv[1], "units") == 0) {
    const int u = units();
    return flow_range_units() == 0 ? u : 1;
  }
  if (argc == 2 && std::strcmp(argv[1], "flow") == 0) return flow();
  std::fprintf(stderr, "usage: host_logic_check units|flow\n");
  return 2;
}
