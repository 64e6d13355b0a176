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
#include <vector>

#include "fd_linalg.hpp"
#include "fd_solver.hpp"

namespace fd {

constexpr double KAPPA_P = 10.0;   // safety factor of the Perron wall (eq. perronwall)
constexpr double ETA_FP32 = 1e-7;  // precision scale of float32 kernels

struct SolverLayout {
  int b = 0, k = 0, keep = 0, kk = 0, mm = 0;
  bool dense = false;
};

static SolverLayout solver_layout(int64_t N, int b, int k, const fd_lanczos_opts& o) {
  SolverLayout L;
  L.b = b;
  L.k = k;
  L.keep = o.keep >= 0 ? o.keep : b;
  L.kk = k + L.keep;
  int mm = o.max_basis_blocks > 0 ? o.max_basis_blocks * b
                                  : int(round_up(L.kk, b) + std::max<int64_t>(2 * b, round_up(L.kk, b)));
  mm = std::min(mm, (1024 / b) * b);  // projected eigensolve limit
  if (N <= mm) {
    L.dense = true;
    L.mm = int(N);
    L.kk = int(N);
    return L;
  }
  L.mm = mm;
  FD_REQUIRE(L.kk + b <= mm, FD_ERR_INVALID_ARG,
             "basis too small: need k + keep + b <= max_basis_blocks * b (and <= 1024)");
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
  double *T = nullptr, *Tw = nullptr, *S = nullptr, *Vw = nullptr, *theta = nullptr;
  double *C = nullptr, *G = nullptr, *res = nullptr;
  float *C32 = nullptr, *S32 = nullptr, *Rinv = nullptr;
  int *flags = nullptr, *sel = nullptr, *sweeps = nullptr;
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
  if (w.prod.plan.nsplit > 1)
    w.prod.part = a.fspan(size_t(w.prod.plan.nsplit) * w.prod.rows.npad * w.prod.plan.ncb * 16);
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
  w.S = a.take<double>(m2);
  w.Vw = a.take<double>(m2);
  w.theta = a.take<double>(mm_cap);
  w.res = a.take<double>(mm_cap);
  w.C = a.take<double>(size_t(mm_cap) * b);
  w.C32 = a.take<float>(size_t(mm_cap) * std::max(b, 64));
  w.S32 = a.take<float>(size_t(mm_cap) * 64);
  w.G = a.take<double>(size_t(b) * b);
  w.Rinv = a.take<float>(size_t(b) * b);
  w.flags = a.take<int>(64);
  w.sel = a.take<int>(64);
  w.sweeps = a.take<int>(1);
  return w;
}

static int cap_for(int64_t N, int b, int k, const fd_lanczos_opts& o) {
  const SolverLayout L = solver_layout(N, b, k, o);
  return L.mm;
}

void carve_solver(Arena& a, int64_t N, int64_t D, int b, int k, const fd_lanczos_opts& o,
                  bool continuation) {
  // the widest basis any prefix can need is the iterative one (dense bases are
  // at most that wide); continuation also runs a 64-wide Nystrom product
  fd_lanczos_opts big = o;
  const SolverLayout L = solver_layout(N, b, k, big);
  carve_solver_ws(a, N, D, b, L.mm, continuation ? 64 : b);
}

// ----------------------------------------------------------------- solver

struct Lanczos {
  SolverWs& w;
  hipStream_t st;
  int64_t N;
  int b, mm;
  uint64_t seed;
  uint64_t rng_stream = 1;
  int matvecs = 0;
  bool diag = true;

  Lanczos(SolverWs& ws, hipStream_t s, int64_t n, int bb, int m, uint64_t sd)
      : w(ws), st(s), N(n), b(bb), mm(m), seed(sd) {}

  // Y[:, 0:nb] (ld mm) = M V[:, 0:nb] (ld mm)
  void matvec(const float* V, float* Y, int nb) {
    product_apply(w.prod, w.s, w.s, V, mm, nb, Y, mm, diag, st);
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

  // Rayleigh-Ritz on T[0:m, 0:m]: Ritz values (descending) to theta, the
  // leading nkeep Ritz vectors / images to Qa / Wa, their residual norms to res.
  void rayleigh_ritz(int m, int nkeep) {
    copy_square(w.T, mm, w.Tw, mm, m, st);
    jacobi_eig(w.Tw, m, mm, w.Vw, w.theta, w.S, mm, w.sweeps, st);
    for (int c0 = 0; c0 < nkeep; c0 += 64) {
      const int nc = std::min(64, nkeep - c0);
      narrow(w.S + c0, mm, m, nc, w.S32, st);
      gemm_nn(w.Q, mm, m, w.S32, nc, w.Qa + c0, mm, N, 1.f, 0.f, st);
      gemm_nn(w.W, mm, m, w.S32, nc, w.Wa + c0, mm, N, 1.f, 0.f, st);
    }
    residual_norms(w.Qa, w.Wa, mm, nkeep, w.theta, N, w.part, w.res, st);
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
                                 const fd_lanczos_opts& o) {
  hipStream_t st = L.st;
  const int64_t N = L.N;
  const int b = lay.b, mm = lay.mm;
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
  while (true) {
    const bool full = lay.dense || m + b > mm;
    const bool out_of_budget = L.matvecs >= budget;
    if (full || need_rr || out_of_budget) {
      const int nkeep = lay.dense ? std::min(mm, std::max(k, 1)) : std::min(lay.kk, m);
      L.rayleigh_ritz(m, nkeep);
      FD_HIP_CHECK(hipMemcpyAsync(th.data(), w.theta, sizeof(double) * m, hipMemcpyDeviceToHost, st));
      FD_HIP_CHECK(hipMemcpyAsync(rs.data(), w.res, sizeof(double) * nkeep, hipMemcpyDeviceToHost, st));
      FD_HIP_CHECK(hipStreamSynchronize(st));
      std::swap(w.Q, w.Qa);
      std::swap(w.W, w.Wa);
      int nconv = 0;
      while (nconv < k && rs[nconv] <= o.tol) ++nconv;
      R.nconv = nconv;
      R.theta.assign(th.begin(), th.begin() + std::min(m, std::max(k, 2)));
      R.res.assign(rs.begin(), rs.begin() + std::min(nkeep, k));
      if (nconv >= k || lay.dense) {
        R.converged = nconv >= k;
        break;
      }
      if (out_of_budget || R.restarts >= o.max_restarts) break;
      if (!need_rr) ++R.restarts;
      need_rr = false;
      // restart: keep the Ritz pairs, next block from the leading unconverged residuals
      m = nkeep;
      set_diag(w.T, mm, mm, w.theta, m, st);
      int ns = 0;
      for (int c = 0; c < nkeep && ns < b; ++c)
        if (rs[c] > o.tol) sel[ns++] = c;
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
                      int k) {
  if (info == nullptr) return;
  info->restarts = R.restarts;
  info->block_matvecs = R.matvecs;
  info->nconv = R.nconv;
  double gap = 0.0;
  if (R.theta.size() >= 2 && R.theta[0] != 0.0) gap = (R.theta[0] - R.theta[1]) / std::fabs(R.theta[0]);
  info->gap_perron = gap;
  info->wall = gap <= KAPPA_P * ETA_FP32 ? 1 : 0;
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
      carve_solver(m, N, D, int(b), int(k), o, false);
      check_workspace(ws, ws_bytes, m.used);
      Arena a;
      a.base = static_cast<char*>(ws);
      a.cap = ws_bytes;
      SolverWs w = carve_solver_ws(a, N, D, int(b), lay.mm, int(b));
      hipStream_t st = static_cast<hipStream_t>(stream);

      degree_run(w.deg, X, xt, N, D, ldx, beta, alpha, nullptr, w.d, w.s, w.s_off, true, st);
      Lanczos L(w, st, N, int(b), lay.mm, o.seed);
      SolveResult R = lanczos_solve(w, L, lay, int(k), V0, V0 ? k0 : 0, ldv0,
                                    warm_is_psi ? 0.5 : 0.0, o);
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
      fill_info(info, R, s_off, secs, int(k));
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

fd_status fd_continuation(const void*, fd_dtype, int64_t, int64_t, int64_t, float, const int64_t*,
                          const float*, int64_t, int64_t, int64_t, const float*, int64_t, int64_t,
                          const fd_lanczos_opts*, double*, float*, float*, fd_lanczos_info*,
                          int32_t, int64_t*, void*, size_t, void*) {
  set_error("continuation not built yet");
  return FD_ERR_UNSUPPORTED;
}

}  // extern "C"
