// Block Lanczos eigensolver of M = diag(s) K diag(s) and the (n, beta)
// continuation built on it (FlashDiffusion Sec. 2.3; Sec. 1, last paragraph).
//
// Method.  The paper names block implicitly restarted Lanczos.  This is the
// thick-restart form of it (mathematically equivalent to implicit restarts
// with exact shifts) with full reorthogonalisation:
//   * the basis Q (N x m, orthonormal columns) and its images W = M Q are kept
//     explicitly, and T = Q^T W is assembled from exact inner products, so the
//     Rayleigh-Ritz step and the residuals ||M y - theta y|| are true values
//     for any starting subspace (also a warm start that is not a Krylov block);
//   * expansion: the images of the newest block are orthogonalised against the
//     whole basis twice (classical Gram-Schmidt, twice) and orthonormalised by
//     Cholesky QR with dependent columns replaced by random ones; one fused
//     product gives their images;
//   * restart (basis full): Rayleigh-Ritz on T (float64 Jacobi on the device),
//     the leading kk Ritz vectors and their images are kept, and the next block
//     is spanned by the residuals of the leading unconverged Ritz pairs (for a
//     Krylov basis these all lie in the one block a Lanczos step would add).
// Small problems (N no larger than the basis) are solved in the full space.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <vector>

#include "fd_host_logic.hpp"
#include "fd_linalg.hpp"
#include "fd_solver.hpp"

namespace fd {

using logic::at_perron_wall;
using logic::count_converged;
using logic::eta_of;
using logic::KAPPA_P;
using logic::next_cycle_width;
using logic::restart_columns;
using logic::SolverLayout;

static SolverLayout solver_layout(int64_t N, int b, int k, const fd_lanczos_opts& o) {
  SolverLayout L;
  const std::string why = logic::solver_layout(N, b, k, o.keep, o.max_basis_blocks, L);
  FD_REQUIRE(why.empty(), FD_ERR_INVALID_ARG, why);
  return L;
}

// Device regions of the eigensolver.
struct SolverWs {
  DegreeWs deg;
  ProductWs prod;
  float *d = nullptr, *s = nullptr;
  double* s_off = nullptr;
  float *Q = nullptr, *Qa = nullptr, *W = nullptr, *Wa = nullptr, *Zt = nullptr;
  FSpanD part;
  double *T = nullptr, *Tw = nullptr, *Tw2 = nullptr, *S = nullptr, *Vw = nullptr,
         *theta = nullptr, *norms = nullptr;
  FSpanD jlog;
  double *C = nullptr, *G = nullptr, *res = nullptr;
  float *C32 = nullptr, *S32 = nullptr, *Rinv = nullptr, *L32 = nullptr;
  double* orth = nullptr;
  int *flags = nullptr, *sel = nullptr, *sweeps = nullptr, *jstate = nullptr;
  int64_t N = 0;
  int mm_cap = 0, b = 0;
};

// prod_width: widest product the caller will run (b, or 64 for the Nystrom pass)
static SolverWs carve_solver_ws(Arena& a, int64_t N, int64_t D, int b, int mm_cap,
                                int prod_width) {
  SolverWs w;
  w.N = N;
  w.mm_cap = mm_cap;
  w.b = b;
  w.deg = carve_degree(a, N, D);
  // the product shares the degree pass's point packs
  w.prod.plan = plan_product(N, N, padded_dim(D), prod_width);
  w.prod.rows = w.deg.rows;
  w.prod.cols = w.deg.cols;
  w.prod.vp = a.fspan(size_t(w.prod.cols.npad) * w.prod.plan.ncb * 16);
  w.prod.vscale = a.fspan(128);
  w.prod.part = a.fspan(part_rows_bound(w.prod.rows.npad, N) * w.prod.plan.ncb * 16);
  w.prod.tmp = a.fspan(size_t(N));  // single-column products (block width 1)
  w.d = a.take<float>(size_t(N));
  w.s = a.take<float>(size_t(N));
  w.s_off = a.take<double>(1);
  const size_t nq = size_t(N) * mm_cap;
  w.Q = a.take<float>(nq);
  w.Qa = a.take<float>(nq);
  w.W = a.take<float>(nq);
  w.Wa = a.take<float>(nq);
  w.Zt = a.take<float>(size_t(N) * b);
  const size_t part_gemm = size_t(gemm_tn_chunks(N)) * mm_cap * std::max(b, 1);
  const size_t part_res = size_t(64) * mm_cap;
  w.part = take_d(a, std::max(part_gemm, part_res));
  const size_t m2 = size_t(mm_cap) * mm_cap;
  w.T = a.take<double>(m2);
  w.Tw = a.take<double>(m2);
  w.Tw2 = a.take<double>(m2);
  w.norms = a.take<double>(2);
  w.S = a.take<double>(m2);
  w.Vw = a.take<double>(m2);
  w.jlog = take_d(a, jacobi_log_doubles(mm_cap));
  w.theta = a.take<double>(mm_cap);
  w.res = a.take<double>(mm_cap);
  w.C = a.take<double>(size_t(mm_cap) * b);
  w.C32 = a.take<float>(size_t(mm_cap) * std::max(b, 64));
  w.S32 = a.take<float>(size_t(mm_cap) * 64);
  w.L32 = a.take<float>(size_t(mm_cap) * mm_cap);
  w.orth = a.take<double>(1);
  w.G = a.take<double>(size_t(b) * b);
  w.Rinv = a.take<float>(size_t(b) * b);
  w.flags = a.take<int>(64);
  w.sel = a.take<int>(64);
  w.sweeps = a.take<int>(1);
  w.jstate = a.take<int>(2);
  return w;
}

void carve_solver(Arena& a, int64_t N, int64_t D, int b, int k, const fd_lanczos_opts& o) {
  const SolverLayout L = solver_layout(N, b, k, o);
  carve_solver_ws(a, N, D, b, L.mm, b);
}

// ----------------------------------------------------------------- solver

struct Lanczos {
  SolverWs& w;
  ProductWs prod;  // product view for the current number of points
  hipStream_t st;
  int64_t N;
  int b, mm;
  uint64_t seed;
  uint64_t rng_stream = 1;
  int matvecs = 0;
  bool diag = true;

  Lanczos(SolverWs& ws, const ProductWs& pv, hipStream_t s, int64_t n, int bb, int m, uint64_t sd)
      : w(ws), prod(pv), st(s), N(n), b(bb), mm(m), seed(sd) {}

  // Y[:, 0:nb] (ld mm) = M V[:, 0:nb] (ld mm)
  void matvec(const float* V, float* Y, int nb) {
    product_apply(prod, w.s, w.s, V, mm, nb, Y, mm, diag, st);
    ++matvecs;
  }

  // Z[:, 0:nb] (ld mm) <- orthonormal, orthogonal to Q[:, 0:m]
  void cgs2(float* Z, int nb, int m) {
    if (m == 0) return;
    for (int pass = 0; pass < 2; ++pass) {
      gemm_tn(w.Q, mm, m, Z, mm, nb, N, w.part, nullptr, w.C32, st);
      gemm_nn(w.Q, mm, m, w.C32, nb, Z, mm, N, -1.f, 1.f, st);
    }
  }
  void cgs2_t(float* Z, int64_t ldz, int nb, int m) {
    if (m == 0) return;
    for (int pass = 0; pass < 2; ++pass) {
      gemm_tn(w.Q, mm, m, Z, ldz, nb, N, w.part, nullptr, w.C32, st);
      gemm_nn(w.Q, mm, m, w.C32, nb, Z, ldz, N, -1.f, 1.f, st);
    }
  }
  void orth_block(float* Z, int nb, int m) {
    cgs2(Z, nb, m);
    gemm_tn(Z, mm, nb, Z, mm, nb, N, w.part, w.G, nullptr, st);
    chol_rinv(w.G, nb, 1e-4, w.Rinv, w.flags, st);
    gemm_nn(Z, mm, nb, w.Rinv, nb, w.Zt, nb, N, 1.f, 0.f, st);
    fill_normal(w.Zt, nb, N, nb, w.flags, seed, rng_stream++, st);
    cgs2_t(w.Zt, nb, nb, m);
    gemm_tn(w.Zt, nb, nb, w.Zt, nb, nb, N, w.part, w.G, nullptr, st);
    chol_rinv(w.G, nb, 1e-4, w.Rinv, w.flags, st);
    gemm_nn(w.Zt, nb, nb, w.Rinv, nb, Z, mm, N, 1.f, 0.f, st);
  }

  // images of Q[:, c0:c0+nb] and the matching rows / columns of T
  void image_block(int c0, int nb) {
    matvec(w.Q + c0, w.W + c0, nb);
    const int m = c0 + nb;
    gemm_tn(w.Q, mm, m, w.W + c0, mm, nb, N, w.part, w.C, nullptr, st);
    put_block(w.T, mm, w.C, m, c0, nb, st);
  }

  // Thick restart on the kept Ritz pairs Q[:, 0:kk], W[:, 0:kk]: they are
  // re-orthonormalised (first-order Loewdin: Q <- Q (3 I - G) / 2 with
  // G = Q^T Q, W by the same factor) and their block of T is the projection
  // Q^T W itself.  Without this the float32 products Q S of every restart
  // let Q^T Q drift from I over many restarts, and T = diag(theta) (which
  // assumes it) then stalls the residuals near the tolerance.  Qa, Wa are
  // scratch here.
  void refresh_kept(int kk) {
    for (int c0 = 0; c0 < kk; c0 += b) {
      const int nc = std::min(b, kk - c0);
      gemm_tn(w.Q, mm, kk, w.Q + c0, mm, nc, N, w.part, w.C, nullptr, st);
      put_block(w.Tw, mm, w.C, kk, c0, nc, st);
    }
    loewdin(w.Tw, mm, kk, 64, w.L32, w.orth, st);
    for (int c0 = 0; c0 < kk; c0 += 64) {
      const int nc = std::min(64, kk - c0);
      gemm_nn(w.Q, mm, kk, w.L32 + int64_t(kk) * c0, nc, w.Qa + c0, mm, N, 1.f, 0.f, st);
      gemm_nn(w.W, mm, kk, w.L32 + int64_t(kk) * c0, nc, w.Wa + c0, mm, N, 1.f, 0.f, st);
    }
    std::swap(w.Q, w.Qa);
    std::swap(w.W, w.Wa);
    set_diag(w.T, mm, mm, nullptr, 0, st);
    for (int c0 = 0; c0 < kk; c0 += b) {
      const int nc = std::min(b, kk - c0);
      gemm_tn(w.Q, mm, kk, w.W + c0, mm, nc, N, w.part, w.C, nullptr, st);
      put_block(w.T, mm, w.C, kk, c0, nc, st);
    }
  }

  // Rayleigh-Ritz on T[0:m, 0:m]: Ritz values (descending) to theta, the
  // leading nkeep Ritz vectors / images to Qa / Wa, their residual norms to res.
  int rayleigh_ritz(int m, int nkeep) {
    copy_square(w.T, mm, w.Tw, mm, m, st);
    const int sweeps = jacobi_eig(w.Tw, w.Tw2, m, mm, w.Vw, w.theta, w.S, mm, w.norms, w.jlog, w.jstate, st);
    for (int c0 = 0; c0 < nkeep; c0 += 64) {
      const int nc = std::min(64, nkeep - c0);
      narrow(w.S + c0, mm, m, nc, w.S32, st);
      gemm_nn(w.Q, mm, m, w.S32, nc, w.Qa + c0, mm, N, 1.f, 0.f, st);
      gemm_nn(w.W, mm, m, w.S32, nc, w.Wa + c0, mm, N, 1.f, 0.f, st);
    }
    residual_norms(w.Qa, w.Wa, mm, nkeep, w.theta, N, w.part, w.res, st);
    return sweeps;
  }
};

struct SolveResult {
  std::vector<double> theta, res;
  int restarts = 0, matvecs = 0, nconv = 0;
  bool converged = false;
};

// Solve on the first N points of the packed set.  The normalisation (d, s)
// must already be in w.d / w.s.  On return Q[:, 0:k] (ld mm) holds the Ritz
// vectors.  V0 (optional) is copied in as the start (ld ldv0, k0 columns),
// scaled by d^scale_pow (0.5 turns Markov vectors into M's).
static SolveResult lanczos_solve(SolverWs& w, Lanczos& L, const SolverLayout& lay, int k,
                                 const float* V0, int64_t k0, int64_t ldv0, double scale_pow,
                                 const fd_lanczos_opts& o, double eta) {
  hipStream_t st = L.st;
  const int64_t N = L.N;
  const int b = lay.b, mm = lay.mm;
  const auto t_start = std::chrono::steady_clock::now();
  SolveResult R;
  int m = 0;
  bool need_rr = false;

  if (lay.dense) {
    set_identity(w.Q, mm, N, mm, st);
    for (int c0 = 0; c0 < mm; c0 += b) {
      const int nb = std::min(b, mm - c0);
      L.image_block(c0, nb);
    }
    m = mm;
    need_rr = true;
  } else {
    int n0 = b;
    int kw = 0;
    if (V0 != nullptr && k0 > 0) {
      kw = int(std::min<int64_t>(k0, lay.mm - b));
      n0 = int(round_up(kw, b));
      copy_cols(V0, ldv0, w.Q, mm, N, kw, scale_pow != 0.0 ? w.d : nullptr, scale_pow, st);
      need_rr = true;
    }
    if (n0 > kw) fill_normal(w.Q + kw, mm, N, n0 - kw, nullptr, L.seed, 0, st);
    for (int c0 = 0; c0 < n0; c0 += b) L.orth_block(w.Q + c0, b, c0);
    for (int c0 = 0; c0 < n0; c0 += b) L.image_block(c0, b);
    m = n0;
  }

  std::vector<double> th(mm), rs(mm);
  std::vector<int> sel(b);
  const int budget = o.max_matvecs > 0 ? o.max_matvecs : INT32_MAX;
  int width = lay.m_first;  // basis width of the current restart cycle
  int nconv_cycle = 0;      // leading converged pairs at the last restart
  while (true) {
    const bool full = lay.dense || m + b > width;
    const bool out_of_budget = L.matvecs >= budget;
    if (full || need_rr || out_of_budget) {
      const int nkeep = lay.dense ? std::min(mm, std::max(k, 1)) : std::min(lay.kk, m);
      const int sweeps = L.rayleigh_ritz(m, nkeep);
      FD_HIP_CHECK(hipMemcpyAsync(th.data(), w.theta, sizeof(double) * m, hipMemcpyDeviceToHost, st));
      FD_HIP_CHECK(hipMemcpyAsync(rs.data(), w.res, sizeof(double) * nkeep, hipMemcpyDeviceToHost, st));
      FD_HIP_CHECK(hipStreamSynchronize(st));
      const int nconv = count_converged(rs.data(), k, o.tol);
      if (o.verbose) {
        double worst = 0.0;
        for (int c = 0; c < std::min(k, nkeep); ++c) worst = std::max(worst, rs[c]);
        const double el =
            std::chrono::duration<double>(std::chrono::steady_clock::now() - t_start).count();
        std::fprintf(stderr,
                     "[fd_lanczos] N=%lld cycle=%d basis=%d products=%d converged=%d/%d "
                     "max_residual=%.3e theta0=%.9f theta_k-1=%.6e jacobi_sweeps=%d "
                     "elapsed=%.3fs\n",
                     (long long)N, R.restarts, m, L.matvecs, nconv, k, worst, th[0],
                     th[std::min(k, m) - 1], sweeps, el);
        std::fflush(stderr);
      }
      R.nconv = nconv;
      R.theta.assign(th.begin(), th.begin() + std::min(m, std::max(k, 2)));
      R.res.assign(rs.begin(), rs.begin() + std::min(nkeep, k));
      const bool done = nconv >= k || lay.dense;
      const bool at_wall = at_perron_wall(m, th[0], m >= 2 ? th[1] : 0.0, rs[0], o.tol, eta);
      const bool stop = out_of_budget || R.restarts >= o.max_restarts || at_wall;
      // the leading Ritz vectors and their images become the basis
      std::swap(w.Q, w.Qa);
      std::swap(w.W, w.Wa);
      if (done) {
        R.converged = nconv >= k;
        break;
      }
      if (stop) break;
      if (!need_rr) {
        ++R.restarts;
        width = next_cycle_width(lay, width, nconv_cycle, nconv);
      } else {
        width = logic::warm_cycle_width(lay, nkeep);
      }
      nconv_cycle = nconv;
      need_rr = false;
      // restart: keep the Ritz pairs, next block from the leading unconverged residuals
      m = nkeep;
      L.refresh_kept(m);
      if (o.verbose) {
        double dev = 0.0;
        FD_HIP_CHECK(hipMemcpyAsync(&dev, w.orth, sizeof(dev), hipMemcpyDeviceToHost, st));
        FD_HIP_CHECK(hipStreamSynchronize(st));
        std::fprintf(stderr, "[fd_lanczos] N=%lld restart: kept basis max|Q^T Q - I| = %.3e\n",
                     (long long)N, dev);
        std::fflush(stderr);
      }
      const int ns = restart_columns(rs.data(), nkeep, b, o.tol, sel.data());
      FD_HIP_CHECK(hipMemcpyAsync(w.sel, sel.data(), sizeof(int) * ns, hipMemcpyHostToDevice, st));
      float* Z = w.Q + m;
      gather_residuals(w.Q, w.W, mm, w.theta, w.sel, ns, Z, mm, N, st);
      if (ns < b) fill_normal(Z + ns, mm, N, b - ns, nullptr, L.seed, L.rng_stream++, st);
      L.orth_block(Z, b, m);
      L.image_block(m, b);
      m += b;
      // the host vectors must stay alive until the copy ran
      FD_HIP_CHECK(hipStreamSynchronize(st));
      continue;
    }
    // expansion from the images of the newest block
    float* Z = w.Q + m;
    copy_cols(w.W + (m - b), mm, Z, mm, N, b, nullptr, 0.0, st);
    L.orth_block(Z, b, m);
    L.image_block(m, b);
    m += b;
  }
  R.matvecs = L.matvecs;
  return R;
}

static void fill_info(fd_lanczos_info* info, const SolveResult& R, double s_off, double secs,
                      int k, double eta) {
  if (info == nullptr) return;
  info->restarts = R.restarts;
  info->block_matvecs = R.matvecs;
  info->nconv = R.nconv;
  const double gap = R.theta.size() >= 2 ? logic::perron_gap(R.theta[0], R.theta[1]) : 0.0;
  info->gap_perron = gap;
  info->wall = gap <= KAPPA_P * eta ? 1 : 0;
  info->s_off = s_off;
  double mx = 0.0;
  for (int i = 0; i < k && i < int(R.res.size()); ++i) mx = std::max(mx, R.res[i]);
  info->max_residual = mx;
  info->seconds = secs;
}

static void validate_opts(const fd_lanczos_opts& o) {
  FD_REQUIRE(std::isfinite(o.tol) && o.tol > 0.0, FD_ERR_INVALID_ARG, "tol must be > 0");
  FD_REQUIRE(o.max_restarts >= 0 && o.max_matvecs >= 0 && o.max_basis_blocks >= 0,
             FD_ERR_INVALID_ARG, "negative option");
}

// ----------------------------------------------------------------- continuation

struct ContWs {
  SolverWs sw;
  float* store_psi = nullptr;  // nsteps x (nmax x k): Markov vectors of every step
  float* store_q = nullptr;    // nsteps x nmax: degrees q of every step
  float* ext = nullptr;        // nmax x k: Nystrom-extended start
  float* den = nullptr;        // nmax: K w of the extension
  float* wv = nullptr;         // nmax: w = q^-alpha of the source step
  float* num = nullptr;        // nmax x 64: K (w psi) of the extension
  double* lam = nullptr;       // k: source eigenvalues
  int64_t nmax = 0;
  int k = 0;
  float* psi(int64_t t) const { return store_psi + size_t(t) * nmax * k; }
  float* q(int64_t t) const { return store_q + size_t(t) * nmax; }
};

static ContWs carve_continuation(Arena& a, int64_t nmax, int64_t nsteps, int64_t D, int b, int k,
                                 const fd_lanczos_opts& o) {
  ContWs c;
  c.nmax = nmax;
  c.k = k;
  const SolverLayout L = solver_layout(nmax, b, k, o);
  c.sw = carve_solver_ws(a, nmax, D, b, L.mm, 64);
  c.store_psi = a.take<float>(size_t(nsteps) * nmax * k);
  c.store_q = a.take<float>(size_t(nsteps) * nmax);
  c.ext = a.take<float>(size_t(nmax) * k);
  c.den = a.take<float>(size_t(nmax));
  c.wv = a.take<float>(size_t(nmax));
  c.num = a.take<float>(size_t(nmax) * 64);
  c.lam = a.take<double>(64);
  return c;
}

// ext[i, c] = (1/lambda_c) sum_j K_ij w_j psi_jc / sum_j K_ij w_j
__global__ void nystrom_finish_kernel(const float* __restrict__ num, int ldn,
                                      const float* __restrict__ den,
                                      const double* __restrict__ lam, int64_t n, int c0, int nc,
                                      float* __restrict__ ext, int lde) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= n * nc) return;
  const int64_t i = idx / nc;
  const int c = int(idx % nc);
  ext[i * lde + c0 + c] = float(double(num[i * ldn + c]) / double(den[i]) / lam[c0 + c]);
}

// Extend Markov vectors psi (n_old x k, ld k) of the step solved at beta on the
// prefix n_old to the prefix n_new by the Nystrom extension the paper uses to
// warm-start a larger nested sample (Sec. 1, last paragraph; Sec. 2.3, dyadic
// continuation).  The paper names the extension without a formula; the one
// here is the eigen-relation P psi = lambda psi evaluated at a new point:
//   psi(x) = (1 / lambda) sum_j K(x, x_j) w_j psi_j / sum_j K(x, x_j) w_j,
// w = q^-alpha of the old sample (the new point's own q^-alpha cancels).
// One row-sum pass gives the denominators, ceil(k / 64) fused products the
// numerators.
static void nystrom_extend(ContWs& c, const void* X, fd_dtype xt, int64_t D, int64_t ldx,
                           int64_t n_old, int64_t n_new, double beta, double alpha,
                           const float* psi, const float* q_old, const std::vector<double>& lam,
                           int k, hipStream_t st) {
  SolverWs& w = c.sw;
  PointPack rows = pack_view(w.deg.rows, n_new, ROW_PAD);
  PointPack cols = pack_view(w.deg.cols, n_old, COL_PAD);
  // centred on the old prefix (the column set), radius over the new one
  launch_centre(X, xt, n_old, D, ldx, w.deg.centre, st);
  launch_radius_more(X, xt, n_new, D, ldx, w.deg.centre, st);
  launch_pack_points(X, xt, n_new, D, ldx, beta, true, rows, &w.deg.centre, st);
  launch_pack_points(X, xt, n_old, D, ldx, beta, false, cols, &w.deg.centre, st);
  launch_pow_neg(q_old, n_old, alpha, c.wv, st);
  // denominators K w
  launch_pack_w(c.wv, n_old, cols.npad, w.deg.wp, st);
  KVPlan rp = plan_rowsum(n_new, n_old, rows.dp);
  launch_rowsum(rp, rows, cols, w.deg.wp, true, c.den, w.deg.part, st);
  // numerators K (w psi), 64 columns at a time
  std::vector<double> l(lam.begin(), lam.begin() + k);
  FD_HIP_CHECK(hipMemcpyAsync(c.lam, l.data(), sizeof(double) * k, hipMemcpyHostToDevice, st));
  ProductWs pv = product_view(w.prod, rows, cols, 64);
  for (int c0 = 0; c0 < k; c0 += 64) {
    const int nc = std::min(64, k - c0);
    product_apply(pv, nullptr, c.wv, psi + c0, k, nc, c.num, 64, true, st);
    hipLaunchKernelGGL(nystrom_finish_kernel, dim3(unsigned((n_new * nc + 255) / 256)), dim3(256),
                       0, st, c.num, 64, c.den, c.lam, n_new, c0, nc, c.ext, k);
    FD_LAUNCH_CHECK();
  }
  FD_HIP_CHECK(hipStreamSynchronize(st));
}

void carve_continuation_ws(Arena& a, int64_t nmax, int64_t nsteps, int64_t D, int b, int k,
                           const fd_lanczos_opts& o) {
  carve_continuation(a, nmax, nsteps, D, b, k, o);
}

// ----------------------------------------------------------------- bandwidth flow
//
// Sec. 2.3 ("beta-function flow"): dyadic probes from beta_0, the empirical
// potential V = V_bias + V_stat + V_mach over log beta, the bracketing rule
// with a quadratic vertex probe, and the Perron wall.

struct FlowWs {
  SolverWs sw;
  float* psi_keep = nullptr;  // N x k: Markov vectors of the latest admissible probe
  float* psi_new = nullptr;   // N x k: Markov vectors of the probe being solved
  double* stats = nullptr;    // centring: nblk x (D + 1) partials, D means, 1 total
  int nblk = 0;
};

static int flow_stat_blocks(int64_t N) {
  return int(std::min<int64_t>(256, std::max<int64_t>(1, (N + 4095) / 4096)));
}

static FlowWs carve_flow(Arena& a, int64_t N, int64_t D, int b, int k, const fd_lanczos_opts& o) {
  FlowWs f;
  const SolverLayout L = solver_layout(N, b, k, o);
  f.sw = carve_solver_ws(a, N, D, b, L.mm, b);
  f.psi_keep = a.take<float>(size_t(N) * k);
  f.psi_new = a.take<float>(size_t(N) * k);
  f.nblk = flow_stat_blocks(N);
  f.stats = a.take<double>(size_t(f.nblk) * (D + 1) + size_t(D) + 1);
  return f;
}

void carve_flow_ws(Arena& a, int64_t N, int64_t D, int b, int k, const fd_lanczos_opts& o) {
  carve_flow(a, N, D, b, k, o);
}

__device__ __forceinline__ double x_at(const float* X, int64_t i) { return double(X[i]); }
__device__ __forceinline__ double x_at(const uint16_t* X, int64_t i) {
  return double(__uint_as_float(uint32_t(X[i]) << 16));
}

// Block partials over rows [blk rpb, (blk + 1) rpb), fixed order: the column
// sums (mu == NULL) or sum_i ||x_i - mu||^2 (mu given, into slot D).
template <typename T>
__global__ __launch_bounds__(256) void centre_partial_kernel(const T* __restrict__ X, int64_t N,
                                                             int D, int64_t ldx,
                                                             const double* __restrict__ mu,
                                                             int64_t rpb,
                                                             double* __restrict__ part) {
  __shared__ double red[256];
  const int t = threadIdx.x;
  const int64_t r0 = int64_t(blockIdx.x) * rpb;
  const int64_t r1 = min(N, r0 + rpb);
  const int nout = mu == nullptr ? D : 1;
  for (int k = 0; k < nout; ++k) {
    double acc = 0.0;
    for (int64_t i = r0 + t; i < r1; i += 256) {
      if (mu == nullptr) {
        acc += x_at(X, i * ldx + k);
      } else {
        double r = 0.0;
        for (int f = 0; f < D; ++f) {
          const double v = x_at(X, i * ldx + f) - mu[f];
          r += v * v;
        }
        acc += r;
      }
    }
    red[t] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if (t < w) red[t] += red[t + w];
      __syncthreads();
    }
    if (t == 0) part[int64_t(blockIdx.x) * (D + 1) + (mu == nullptr ? k : D)] = red[0];
    __syncthreads();
  }
}

// out[c] = (sum over blocks of part[., slot0 + c]) / N, c < nc, blocks in order
__global__ void centre_finish_kernel(const double* __restrict__ part, int nblk, int D, int slot0,
                                     int nc, int64_t N, double* __restrict__ out) {
  const int c = threadIdx.x;
  if (c >= nc) return;
  double acc = 0.0;
  for (int b = 0; b < nblk; ++b) acc += part[int64_t(b) * (D + 1) + slot0 + c];
  out[c] = acc / double(N);
}

// mean_i ||x_i - mean||^2 in float64, two passes (means, then deviations).
template <typename T>
static double centred_mean_sq(FlowWs& f, const T* X, int64_t N, int64_t D, int64_t ldx,
                              hipStream_t st) {
  const int64_t rpb = (N + f.nblk - 1) / f.nblk;
  double* part = f.stats;
  double* mu = f.stats + size_t(f.nblk) * (D + 1);
  double* tot = mu + D;
  hipLaunchKernelGGL((centre_partial_kernel<T>), dim3(f.nblk), dim3(256), 0, st, X, N, int(D),
                     ldx, nullptr, rpb, part);
  FD_LAUNCH_CHECK();
  hipLaunchKernelGGL(centre_finish_kernel, dim3(1), dim3(64), 0, st, part, f.nblk, int(D), 0,
                     int(D), N, mu);
  FD_LAUNCH_CHECK();
  hipLaunchKernelGGL((centre_partial_kernel<T>), dim3(f.nblk), dim3(256), 0, st, X, N, int(D),
                     ldx, mu, rpb, part);
  FD_LAUNCH_CHECK();
  hipLaunchKernelGGL(centre_finish_kernel, dim3(1), dim3(64), 0, st, part, f.nblk, int(D),
                     int(D), 1, N, tot);
  FD_LAUNCH_CHECK();
  double ms = 0.0;
  FD_HIP_CHECK(hipMemcpyAsync(&ms, tot, sizeof(double), hipMemcpyDeviceToHost, st));
  FD_HIP_CHECK(hipStreamSynchronize(st));
  return ms;
}

using logic::FlowOutcome;
using logic::FlowParams;
using logic::FlowProbe;

// One probe: normalisation and top-k eigensolve at beta (warm: Markov vectors
// N x k or NULL); the Ritz vectors stay in sw.Q, psi goes to psi_out.
static FlowProbe flow_probe(FlowWs& f, const void* X, fd_dtype xt, int64_t N, int64_t D,
                            int64_t ldx, double beta, double alpha, int b, int k,
                            const float* warm, float* psi_out, const fd_lanczos_opts& o,
                            const FlowParams& fp, int role, uint64_t seed_offset,
                            hipStream_t st) {
  const auto t0 = std::chrono::steady_clock::now();
  FlowProbe pr;
  pr.beta = beta;
  pr.role = role;
  degree_run(f.sw.deg, X, xt, N, D, ldx, beta, alpha, nullptr, f.sw.d, f.sw.s, f.sw.s_off, true,
             st);
  const SolverLayout lay = solver_layout(N, b, k, o);
  Lanczos L(f.sw, product_view(f.sw.prod, f.sw.deg.rows, f.sw.deg.cols, b), st, N, b, lay.mm,
            o.seed + seed_offset);
  SolveResult R = lanczos_solve(f.sw, L, lay, k, warm, warm ? k : 0, k, 0.5, o, eta_of(xt));
  copy_cols(f.sw.Q, lay.mm, psi_out, k, N, k, f.sw.d, -0.5, st);
  FD_HIP_CHECK(hipMemcpyAsync(&pr.s_off, f.sw.s_off, sizeof(double), hipMemcpyDeviceToHost, st));
  FD_HIP_CHECK(hipStreamSynchronize(st));
  pr.evals = R.theta;
  pr.converged = R.converged;
  pr.matvecs = R.matvecs;
  pr.nconv = R.nconv;
  logic::probe_stats(pr, k, fp);
  pr.seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  return pr;
}

static fd_flow_probe flow_record(const FlowProbe& p, int level) {
  fd_flow_probe r{};
  r.level = level;
  r.beta = p.beta;
  r.s_off = p.s_off;
  r.gap_perron = p.gap;
  r.v_bias = p.v_bias;
  r.v_mach = p.v_mach;
  r.n_eff = p.n_eff;
  r.v_stat = p.v_stat;
  r.v_total = p.v_total;
  r.d_hat = p.d_hat;
  r.seconds = p.seconds;
  r.role = p.role;
  r.admissible = p.admissible ? 1 : 0;
  r.status = p.converged ? FD_OK : FD_ERR_NOT_CONVERGED;
  r.block_matvecs = p.matvecs;
  r.nconv = p.nconv;
  return r;
}


// beta_0 of eq. beta0 from the centred data: min(0.1, 1 / (2 mean ||x - mean||^2)).
static double flow_beta0(FlowWs& f, const void* X, fd_dtype xt, int64_t N, int64_t D,
                         int64_t ldx, hipStream_t st) {
  const double ms = xt == FD_BF16
                        ? centred_mean_sq(f, static_cast<const uint16_t*>(X), N, D, ldx, st)
                        : centred_mean_sq(f, static_cast<const float*>(X), N, D, ldx, st);
  return ms > 0.0 ? std::min(0.1, 1.0 / (2.0 * ms)) : 0.1;
}

// One sweep of the flow on X from `beta` (Sec. 2.3; the decisions are
// logic::run_flow_logic).  warm: psi_keep already holds Markov vectors to
// start the first probe from.  Records are appended to `out` with the given
// level.  On return with any == true, sw.Q holds the eigenvectors of the solve
// at fin.beta and psi_keep its Markov vectors.
struct DeviceFlowDriver {
  FlowWs& f;
  const void* X;
  fd_dtype xt;
  int64_t N, D, ldx;
  double alpha;
  int bb, kk;
  const FlowParams& fp;
  const fd_lanczos_opts& o;
  int level;
  std::vector<fd_flow_probe>& out;
  hipStream_t st;
  double r2max;  // max ||x - mean||^2 of X (host copy)

  bool in_range(double beta) const { return exponent_in_range(xt, beta, r2max); }
  FlowProbe probe(double beta, int role, int t, bool from_keep) {
    const uint64_t lseed = uint64_t(level) * 1000003u;
    const uint64_t off = role == 0   ? lseed + uint64_t(t) * 7919u
                         : role == 1 ? lseed + 104729u
                                     : lseed + 15485863u;
    return flow_probe(f, X, xt, N, D, ldx, beta, alpha, bb, kk, from_keep ? f.psi_keep : nullptr,
                      f.psi_new, o, fp, role, off, st);
  }
  void accept() { std::swap(f.psi_keep, f.psi_new); }
  void record(const FlowProbe& p, bool replace_last) {
    if (replace_last)
      out.back() = flow_record(p, level);
    else
      out.push_back(flow_record(p, level));
  }
};

static FlowOutcome run_flow(FlowWs& f, const void* X, fd_dtype xt, int64_t N, int64_t D,
                            int64_t ldx, double alpha, int bb, int kk, double beta, bool warm,
                            const FlowParams& fp, const fd_lanczos_opts& o, int max_probes,
                            int level, std::vector<fd_flow_probe>& out, hipStream_t st) {
  // the radius that bounds the exponent range: X's centring is the same for
  // every probe
  launch_centre(X, xt, N, D, ldx, f.sw.deg.centre, st);
  const double r2 = exponent_radius(xt, f.sw.deg.centre, st);
  DeviceFlowDriver drv{f, X, xt, N, D, ldx, alpha, bb, kk, fp, o, level, out, st, r2};
  return logic::run_flow_logic(drv, N, beta, warm, max_probes);
}

// Status and message of a sweep that produced nothing admissible.
static fd_status flow_nothing_admissible(const FlowOutcome& R, int level, int32_t* exit_reason) {
  const std::string of = level < 0 ? std::string() : " of cascade level " + std::to_string(level);
  if (R.reason == FD_FLOW_RANGE) {
    *exit_reason = FD_FLOW_RANGE;
    set_error("the first bandwidth" + of + " is beyond the float32 exponent range " +
              "(beta log2(e) max ||x - mean||^2 > " + std::to_string(HX_EXP_RANGE) + ")");
    return FD_ERR_UNSUPPORTED;
  }
  *exit_reason = FD_FLOW_WALL;
  set_error("the first probe" + of + " is already past the Perron wall (g_P <= kappa_P eta)");
  return FD_ERR_PERRON_WALL;
}

}  // namespace fd

using namespace fd;

extern "C" {

fd_status fd_block_lanczos(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                           float beta, float alpha, int64_t b, int64_t k, const float* V0,
                           int64_t k0, int64_t ldv0, int32_t warm_is_psi,
                           const fd_lanczos_opts* opts, double* evals, float* evecs, float* psi,
                           double* residuals, fd_lanczos_info* info, void* ws, size_t ws_bytes,
                           void* stream) {
  fd_status status = FD_OK;
  fd_status st0 = [&]() -> fd_status {
    try {
      const auto t0 = std::chrono::steady_clock::now();
      check_points(X, xt, N, D, ldx, "X");
      FD_REQUIRE(std::isfinite(beta) && beta > 0.f, FD_ERR_INVALID_ARG, "beta must be finite and > 0");
      FD_REQUIRE(alpha >= 0.f && alpha <= 1.f, FD_ERR_INVALID_ARG, "alpha must be in [0, 1]");
      FD_REQUIRE(b >= 1 && b <= MAX_B, FD_ERR_INVALID_ARG, "b must be in [1, 64]");
      FD_REQUIRE(k >= 1 && k <= N, FD_ERR_INVALID_ARG, "k must be in [1, N]");
      FD_REQUIRE(evals != nullptr && evecs != nullptr, FD_ERR_INVALID_ARG, "evals / evecs NULL");
      FD_REQUIRE(V0 == nullptr || k0 == 0 || (k0 > 0 && ldv0 >= k0), FD_ERR_INVALID_ARG,
                 "bad warm start");
      fd_lanczos_opts o;
      fd_lanczos_default_opts(&o);
      if (opts != nullptr) o = *opts;
      validate_opts(o);
      const SolverLayout lay = solver_layout(N, int(b), int(k), o);
      FD_REQUIRE(lay.dense || k <= lay.kk, FD_ERR_INVALID_ARG, "k too large for the basis");
      Arena m;
      m.measuring = true;
      carve_solver(m, N, D, int(b), int(k), o);
      check_workspace(ws, ws_bytes, m.used);
      Arena a;
      a.base = static_cast<char*>(ws);
      a.cap = ws_bytes;
      SolverWs w = carve_solver_ws(a, N, D, int(b), lay.mm, int(b));
      hipStream_t st = static_cast<hipStream_t>(stream);
      require_finite(X, xt, N, D, ldx, w.deg.flag, st);

      degree_run(w.deg, X, xt, N, D, ldx, beta, alpha, nullptr, w.d, w.s, w.s_off, true, st);
      require_exponent_range(xt, w.deg.centre, beta, st);
      // the product view takes the packs as filled (kind and bandwidth)
      Lanczos L(w, product_view(w.prod, w.deg.rows, w.deg.cols, int(b)), st, N, int(b), lay.mm,
                o.seed);
      SolveResult R = lanczos_solve(w, L, lay, int(k), V0, V0 ? k0 : 0, ldv0,
                                    warm_is_psi ? 0.5 : 0.0, o, eta_of(xt));
      copy_cols(w.Q, lay.mm, evecs, k, N, int(k), nullptr, 0.0, st);
      if (psi != nullptr) copy_cols(w.Q, lay.mm, psi, k, N, int(k), w.d, -0.5, st);
      double s_off = 0.0;
      FD_HIP_CHECK(hipMemcpyAsync(&s_off, w.s_off, sizeof(double), hipMemcpyDeviceToHost, st));
      FD_HIP_CHECK(hipStreamSynchronize(st));
      for (int i = 0; i < k; ++i) evals[i] = i < int(R.theta.size()) ? R.theta[i] : 0.0;
      if (residuals != nullptr)
        for (int i = 0; i < k; ++i) residuals[i] = i < int(R.res.size()) ? R.res[i] : 0.0;
      const double secs =
          std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
      fill_info(info, R, s_off, secs, int(k), eta_of(xt));
      if (!R.converged) {
        set_error("block Lanczos stopped before all k pairs converged (" +
                  std::to_string(R.nconv) + " of " + std::to_string(k) + ")");
        return FD_ERR_NOT_CONVERGED;
      }
      set_error("");
      return FD_OK;
    } catch (const Error& e) {
      set_error(e.msg);
      return e.status;
    } catch (const std::exception& e) {
      set_error(std::string("internal error: ") + e.what());
      return FD_ERR_HIP;
    }
  }();
  status = st0;
  return status;
}

fd_status fd_continuation(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                          float alpha, const int64_t* n_steps, const float* beta_steps,
                          int64_t nsteps, int64_t b, int64_t k, const float* V0, int64_t k0,
                          int64_t ldv0, const fd_lanczos_opts* opts, double* evals,
                          float* evecs, float* psi, fd_lanczos_info* per_step,
                          int32_t stop_at_wall, int64_t* steps_done, void* ws, size_t ws_bytes,
                          void* stream) {
  try {
    check_points(X, xt, N, D, ldx, "X");
    FD_REQUIRE(alpha >= 0.f && alpha <= 1.f, FD_ERR_INVALID_ARG, "alpha must be in [0, 1]");
    FD_REQUIRE(b >= 1 && b <= MAX_B, FD_ERR_INVALID_ARG, "b must be in [1, 64]");
    FD_REQUIRE(nsteps >= 1 && n_steps != nullptr && beta_steps != nullptr, FD_ERR_INVALID_ARG,
               "empty schedule");
    FD_REQUIRE(evals != nullptr && evecs != nullptr, FD_ERR_INVALID_ARG, "evals / evecs NULL");
    FD_REQUIRE(k >= 1 && k <= 64, FD_ERR_INVALID_ARG, "k must be in [1, 64] for the continuation");
    int64_t nmax = 0;
    for (int64_t t = 0; t < nsteps; ++t) {
      FD_REQUIRE(n_steps[t] >= 2 && n_steps[t] <= N, FD_ERR_INVALID_ARG, "n_t out of [2, N]");
      FD_REQUIRE(t == 0 || n_steps[t] >= n_steps[t - 1], FD_ERR_INVALID_ARG,
                 "n_steps must be non-decreasing");
      FD_REQUIRE(std::isfinite(beta_steps[t]) && beta_steps[t] > 0.f, FD_ERR_INVALID_ARG,
                 "beta_t must be finite and > 0");
      FD_REQUIRE(k <= n_steps[t], FD_ERR_INVALID_ARG, "k larger than a prefix");
      nmax = std::max(nmax, n_steps[t]);
    }
    FD_REQUIRE(V0 == nullptr || k0 == 0 || (k0 > 0 && ldv0 >= k0), FD_ERR_INVALID_ARG,
               "bad warm start");
    fd_lanczos_opts o;
    fd_lanczos_default_opts(&o);
    if (opts != nullptr) o = *opts;
    validate_opts(o);
    Arena m;
    m.measuring = true;
    carve_continuation(m, nmax, nsteps, D, int(b), int(k), o);
    check_workspace(ws, ws_bytes, m.used);
    Arena a;
    a.base = static_cast<char*>(ws);
    a.cap = ws_bytes;
    ContWs c = carve_continuation(a, nmax, nsteps, D, int(b), int(k), o);
    hipStream_t st = static_cast<hipStream_t>(stream);
    require_finite(X, xt, nmax, D, ldx, c.sw.deg.flag, st);
    const int kk = int(k);
    std::vector<std::vector<double>> lam(nsteps);
    std::vector<float> level_beta;
    std::vector<int64_t> level_slot;
    int64_t n_prev = 0;
    bool any_unconverged = false;
    int64_t done = 0;
    int64_t last = -1;
    fd_status status = FD_OK;
    for (int64_t t = 0; t < nsteps; ++t) {
      const auto t0 = std::chrono::steady_clock::now();
      const int64_t n = n_steps[t];
      const double beta = beta_steps[t];
      const float* warm = nullptr;
      int64_t warm_ld = 0, warm_k = 0;
      if (t == 0) {
        if (V0 != nullptr && k0 > 0) {
          warm = V0;
          warm_ld = ldv0;
          warm_k = k0;
        }
      } else if (n == n_prev) {
        warm = c.psi(last);
        warm_ld = kk;
        warm_k = kk;
      } else {
        // Nystrom extension of the matching-beta step of the previous prefix
        const int64_t src = logic::nystrom_source(level_beta, level_slot, beta_steps[t], last);
        nystrom_extend(c, X, xt, D, ldx, n_prev, n, beta_steps[src], alpha, c.psi(src), c.q(src),
                       lam[src], kk, st);
        warm = c.ext;
        warm_ld = kk;
        warm_k = kk;
        level_beta.clear();
        level_slot.clear();
      }
      // normalisation and eigensolve on the prefix
      DegreeWs dv = degree_view(c.sw.deg, n);
      degree_run(dv, X, xt, n, D, ldx, beta, alpha, c.q(t), c.sw.d, c.sw.s, c.sw.s_off, true, st);
      require_exponent_range(xt, dv.centre, beta, st);
      const SolverLayout lay = solver_layout(n, int(b), kk, o);
      FD_REQUIRE(lay.mm <= c.sw.mm_cap, FD_ERR_INVALID_ARG, "internal: basis wider than carved");
      ProductWs pv = product_view(c.sw.prod, dv.rows, dv.cols, int(b));
      Lanczos L(c.sw, pv, st, n, int(b), lay.mm, o.seed + uint64_t(t) * 7919u);
      SolveResult R = lanczos_solve(c.sw, L, lay, kk, warm, warm_k, warm_ld, 0.5, o, eta_of(xt));
      copy_cols(c.sw.Q, lay.mm, c.psi(t), kk, n, kk, c.sw.d, -0.5, st);
      double s_off = 0.0;
      FD_HIP_CHECK(hipMemcpyAsync(&s_off, c.sw.s_off, sizeof(double), hipMemcpyDeviceToHost, st));
      FD_HIP_CHECK(hipStreamSynchronize(st));
      lam[t] = R.theta;
      lam[t].resize(kk, 0.0);
      for (int i = 0; i < kk; ++i) evals[t * kk + i] = lam[t][i];
      const double secs =
          std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
      fd_lanczos_info info{};
      fill_info(&info, R, s_off, secs, kk, eta_of(xt));
      if (per_step != nullptr) per_step[t] = info;
      // a step at the Perron wall is reported (info.wall), not failed: its
      // leading eigenspace is not resolvable in X's precision
      any_unconverged = any_unconverged || (!R.converged && !info.wall);
      level_beta.push_back(beta_steps[t]);
      level_slot.push_back(t);
      n_prev = n;
      last = t;
      done = t + 1;
      if (t == nsteps - 1 || (stop_at_wall && info.wall)) {
        copy_cols(c.sw.Q, lay.mm, evecs, kk, n, kk, nullptr, 0.0, st);
        if (psi != nullptr) copy_cols(c.psi(t), kk, psi, kk, n, kk, nullptr, 0.0, st);
        FD_HIP_CHECK(hipStreamSynchronize(st));
      }
      if (stop_at_wall && info.wall) {
        status = FD_ERR_PERRON_WALL;
        break;
      }
    }
    if (steps_done != nullptr) *steps_done = done;
    if (status == FD_ERR_PERRON_WALL) {
      set_error("stopped at the Perron wall after step " + std::to_string(done - 1));
      return status;
    }
    if (any_unconverged) {
      set_error("at least one step short of the Perron wall stopped before all k pairs converged");
      return FD_ERR_NOT_CONVERGED;
    }
    set_error("");
    return FD_OK;
  } catch (const Error& e) {
    set_error(e.msg);
    return e.status;
  } catch (const std::exception& e) {
    set_error(std::string("internal error: ") + e.what());
    return FD_ERR_HIP;
  }
}

void fd_flow_default_opts(fd_flow_opts* o) {
  if (o == nullptr) return;
  *o = fd_flow_opts{};
  o->beta_start = 0.0;
  o->eta = 0.0;
  o->kappa = 10.0;
  o->p = 6.0;
  o->max_probes = 24;
}

fd_status fd_beta_flow(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx, float alpha,
                       int64_t b, int64_t k, const fd_flow_opts* fopts,
                       const fd_lanczos_opts* opts, fd_flow_probe* probes, int64_t* nprobes,
                       double* beta_x, int32_t* exit_reason, double* evals, float* evecs,
                       float* psi, void* ws, size_t ws_bytes, void* stream) {
  try {
    check_points(X, xt, N, D, ldx, "X");
    FD_REQUIRE(alpha >= 0.f && alpha <= 1.f, FD_ERR_INVALID_ARG, "alpha must be in [0, 1]");
    FD_REQUIRE(b >= 1 && b <= MAX_B, FD_ERR_INVALID_ARG, "b must be in [1, 64]");
    FD_REQUIRE(k >= 2 && k <= N, FD_ERR_INVALID_ARG, "k must be in [2, N]");
    FD_REQUIRE(probes != nullptr && nprobes != nullptr && beta_x != nullptr &&
                   exit_reason != nullptr && evals != nullptr && evecs != nullptr,
               FD_ERR_INVALID_ARG, "NULL output");
    fd_flow_opts fo;
    fd_flow_default_opts(&fo);
    if (fopts != nullptr) fo = *fopts;
    FD_REQUIRE(fo.max_probes >= 1 && fo.max_probes <= 64, FD_ERR_INVALID_ARG,
               "max_probes must be in [1, 64]");
    FD_REQUIRE(std::isfinite(fo.kappa) && fo.kappa > 0.0 && std::isfinite(fo.p) && fo.p > 0.0,
               FD_ERR_INVALID_ARG, "kappa and p must be finite and > 0");
    FD_REQUIRE(std::isfinite(fo.beta_start) && std::isfinite(fo.eta), FD_ERR_INVALID_ARG,
               "beta_start and eta must be finite");
    FlowParams fp{fo.eta > 0.0 ? fo.eta : eta_of(xt), fo.kappa, fo.p};
    fd_lanczos_opts o;
    fd_lanczos_default_opts(&o);
    if (opts != nullptr) o = *opts;
    validate_opts(o);
    const SolverLayout lay = solver_layout(N, int(b), int(k), o);
    FD_REQUIRE(lay.dense || k <= lay.kk, FD_ERR_INVALID_ARG, "k too large for the basis");
    Arena m;
    m.measuring = true;
    carve_flow(m, N, D, int(b), int(k), o);
    check_workspace(ws, ws_bytes, m.used);
    Arena a;
    a.base = static_cast<char*>(ws);
    a.cap = ws_bytes;
    FlowWs f = carve_flow(a, N, D, int(b), int(k), o);
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int kk = int(k), bb = int(b);
    require_finite(X, xt, N, D, ldx, f.sw.deg.flag, st);

    double beta = fo.beta_start;
    if (beta <= 0.0) beta = flow_beta0(f, X, xt, N, D, ldx, st);
    std::vector<fd_flow_probe> out;  // records in the order run
    const FlowOutcome R = run_flow(f, X, xt, N, D, ldx, alpha, bb, kk, beta, false, fp, o,
                                   fo.max_probes, 0, out, st);
    if (!R.any) {
      // the first probe is already past the wall or out of range: nothing
      // admissible to return
      for (size_t i = 0; i < out.size(); ++i) probes[i] = out[i];
      *nprobes = int64_t(out.size());
      *beta_x = NAN;
      return flow_nothing_admissible(R, -1, exit_reason);
    }
    const FlowProbe& fin = R.fin;
    const int reason = R.reason;
    // the selected solve's eigenvectors are in sw.Q, its Markov vectors in psi_keep
    const SolverLayout lz = solver_layout(N, bb, kk, o);
    copy_cols(f.sw.Q, lz.mm, evecs, kk, N, kk, nullptr, 0.0, st);
    if (psi != nullptr) copy_cols(f.psi_keep, kk, psi, kk, N, kk, nullptr, 0.0, st);
    FD_HIP_CHECK(hipStreamSynchronize(st));
    for (int i = 0; i < kk; ++i) evals[i] = fin.evals[i];
    for (size_t i = 0; i < out.size(); ++i) probes[i] = out[i];
    *nprobes = int64_t(out.size());
    *beta_x = fin.beta;
    *exit_reason = reason;
    if (!fin.converged) {
      set_error("the eigensolve at the selected bandwidth stopped before all k pairs converged");
      return FD_ERR_NOT_CONVERGED;
    }
    set_error("");
    return FD_OK;
  } catch (const Error& e) {
    set_error(e.msg);
    return e.status;
  } catch (const std::exception& e) {
    set_error(std::string("internal error: ") + e.what());
    return FD_ERR_HIP;
  }
}

fd_status fd_beta_flow_cascade(const void* const* Xs, const fd_dtype* xts, const int64_t* ldxs,
                               int32_t nlevels, int64_t N, int64_t D, float alpha, int64_t b,
                               int64_t k, const fd_flow_opts* fopts, const fd_lanczos_opts* opts,
                               fd_flow_probe* probes, int64_t* nprobes, double* beta_x,
                               int32_t* exit_reason, double* evals, float* evecs, float* psi,
                               void* ws, size_t ws_bytes, void* stream) {
  try {
    FD_REQUIRE(Xs != nullptr && xts != nullptr && ldxs != nullptr && nlevels >= 1 && nlevels <= 4,
               FD_ERR_INVALID_ARG, "the cascade needs 1 to 4 levels");
    for (int l = 0; l < nlevels; ++l) check_points(Xs[l], xts[l], N, D, ldxs[l], "X level");
    FD_REQUIRE(alpha >= 0.f && alpha <= 1.f, FD_ERR_INVALID_ARG, "alpha must be in [0, 1]");
    FD_REQUIRE(b >= 1 && b <= MAX_B, FD_ERR_INVALID_ARG, "b must be in [1, 64]");
    FD_REQUIRE(k >= 2 && k <= N, FD_ERR_INVALID_ARG, "k must be in [2, N]");
    FD_REQUIRE(probes != nullptr && nprobes != nullptr && beta_x != nullptr &&
                   exit_reason != nullptr && evals != nullptr && evecs != nullptr,
               FD_ERR_INVALID_ARG, "NULL output");
    fd_flow_opts fo;
    fd_flow_default_opts(&fo);
    if (fopts != nullptr) fo = *fopts;
    FD_REQUIRE(fo.max_probes >= 1 && fo.max_probes <= 64, FD_ERR_INVALID_ARG,
               "max_probes must be in [1, 64]");
    FD_REQUIRE(std::isfinite(fo.kappa) && fo.kappa > 0.0 && std::isfinite(fo.p) && fo.p > 0.0,
               FD_ERR_INVALID_ARG, "kappa and p must be finite and > 0");
    FD_REQUIRE(std::isfinite(fo.beta_start) && std::isfinite(fo.eta), FD_ERR_INVALID_ARG,
               "beta_start and eta must be finite");
    fd_lanczos_opts o;
    fd_lanczos_default_opts(&o);
    if (opts != nullptr) o = *opts;
    validate_opts(o);
    const SolverLayout lay = solver_layout(N, int(b), int(k), o);
    FD_REQUIRE(lay.dense || k <= lay.kk, FD_ERR_INVALID_ARG, "k too large for the basis");
    Arena m;
    m.measuring = true;
    carve_flow(m, N, D, int(b), int(k), o);
    check_workspace(ws, ws_bytes, m.used);
    Arena a;
    a.base = static_cast<char*>(ws);
    a.cap = ws_bytes;
    FlowWs f = carve_flow(a, N, D, int(b), int(k), o);
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int kk = int(k), bb = int(b);
    for (int l = 0; l < nlevels; ++l)
      require_finite(Xs[l], xts[l], N, D, ldxs[l], f.sw.deg.flag, st);

    std::vector<fd_flow_probe> out;
    FlowOutcome R;
    double beta = fo.beta_start;
    for (int l = 0; l < nlevels; ++l) {
      const void* X = Xs[l];
      const fd_dtype xt = xts[l];
      const FlowParams fp{fo.eta > 0.0 ? fo.eta : eta_of(xt), fo.kappa, fo.p};
      // level 0 starts from beta_0 (or beta_start); every later level from
      // the previous level's achieved bandwidth and Markov vectors
      if (l == 0 && beta <= 0.0) beta = flow_beta0(f, X, xt, N, D, ldxs[l], st);
      R = run_flow(f, X, xt, N, D, ldxs[l], alpha, bb, kk, beta, l > 0, fp, o, fo.max_probes, l,
                   out, st);
      if (!R.any) {
        for (size_t i = 0; i < out.size(); ++i) probes[i] = out[i];
        *nprobes = int64_t(out.size());
        *beta_x = NAN;
        return flow_nothing_admissible(R, l, exit_reason);
      }
      beta = R.fin.beta;
    }
    const FlowProbe& fin = R.fin;
    copy_cols(f.sw.Q, lay.mm, evecs, kk, N, kk, nullptr, 0.0, st);
    if (psi != nullptr) copy_cols(f.psi_keep, kk, psi, kk, N, kk, nullptr, 0.0, st);
    FD_HIP_CHECK(hipStreamSynchronize(st));
    for (int i = 0; i < kk; ++i) evals[i] = fin.evals[i];
    for (size_t i = 0; i < out.size(); ++i) probes[i] = out[i];
    *nprobes = int64_t(out.size());
    *beta_x = fin.beta;
    *exit_reason = R.reason;
    if (!fin.converged) {
      set_error("the eigensolve at the selected bandwidth stopped before all k pairs converged");
      return FD_ERR_NOT_CONVERGED;
    }
    set_error("");
    return FD_OK;
  } catch (const Error& e) {
    set_error(e.msg);
    return e.status;
  } catch (const std::exception& e) {
    set_error(std::string("internal error: ") + e.what());
    return FD_ERR_HIP;
  }
}

}  // extern "C"
