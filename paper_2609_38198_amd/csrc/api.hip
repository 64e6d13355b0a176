// C ABI entry points: argument validation, workspace carving and the
// composition of the kernels into the operations declared in flashdiff.h.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <exception>
#include <mutex>
#include <string>
#include <vector>

#include "fd_internal.hpp"
#include "fd_solver.hpp"

namespace fd {

static thread_local std::string g_err;
void set_error(const std::string& msg) { g_err = msg; }
const char* get_error() { return g_err.c_str(); }

template <class F>
static fd_status guarded(F&& f) {
  try {
    f();
    set_error("");
    return FD_OK;
  } catch (const Error& e) {
    set_error(e.msg);
    return e.status;
  } catch (const std::exception& e) {
    set_error(std::string("internal error: ") + e.what());
    return FD_ERR_HIP;
  } catch (...) {
    set_error("internal error");
    return FD_ERR_HIP;
  }
}

constexpr int64_t MAX_POINTS = int64_t(1) << 30;

void check_points(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                  const char* what) {
  FD_REQUIRE(X != nullptr, FD_ERR_INVALID_ARG, std::string(what) + " is NULL");
  FD_REQUIRE(xt == FD_F32 || xt == FD_BF16, FD_ERR_INVALID_ARG, "unknown dtype");
  FD_REQUIRE(N >= 1 && N <= MAX_POINTS, FD_ERR_INVALID_ARG,
             std::string("number of points of ") + what + " out of range [1, 2^30]");
  FD_REQUIRE(D >= 1, FD_ERR_INVALID_ARG, "D must be >= 1");
  FD_REQUIRE(D <= MAX_D, FD_ERR_UNSUPPORTED, "D above 64 is not supported");
  FD_REQUIRE(ldx >= D, FD_ERR_INVALID_ARG, "ldx must be >= D");
}

void check_workspace(const void* ws, size_t ws_bytes, size_t need) {
  FD_REQUIRE(ws_bytes >= need, FD_ERR_WORKSPACE,
             "workspace too small: need " + std::to_string(need) + " bytes, got " +
                 std::to_string(ws_bytes));
  FD_REQUIRE(need == 0 || ws != nullptr, FD_ERR_WORKSPACE, "workspace is NULL");
  FD_REQUIRE((reinterpret_cast<uintptr_t>(ws) & 255) == 0, FD_ERR_WORKSPACE,
             "workspace must be 256-byte aligned");
}

// ---------------------------------------------------------------- non-finite inputs

__global__ void clear_flag_kernel(int* flag) { *flag = 0; }

__global__ void scan_nonfinite_kernel(const void* __restrict__ X, int bf16, int64_t n, int D,
                                      int64_t ldx, int* __restrict__ flag) {
  const int64_t total = n * D;
  bool bad = false;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
       e += int64_t(gridDim.x) * blockDim.x) {
    const int64_t i = e / D, f = e % D;
    if (bf16) {
      const uint16_t v = static_cast<const uint16_t*>(X)[i * ldx + f];
      bad = bad || (v & 0x7F80u) == 0x7F80u;
    } else {
      bad = bad || !isfinite(static_cast<const float*>(X)[i * ldx + f]);
    }
  }
  if (bad) atomicOr(flag, 1);
}

__global__ void poison_f32_kernel(const int* __restrict__ flag, float* __restrict__ v,
                                  int64_t rows, int64_t cols, int64_t ld) {
  if (*flag == 0) return;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < rows * cols;
       e += int64_t(gridDim.x) * blockDim.x)
    v[(e / cols) * ld + e % cols] = __builtin_nanf("");
}

__global__ void poison_f64_kernel(const int* __restrict__ flag, double* __restrict__ v,
                                  int64_t n) {
  if (*flag == 0) return;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < n;
       e += int64_t(gridDim.x) * blockDim.x)
    v[e] = __builtin_nan("");
}

static unsigned stride_grid(int64_t n) {
  return unsigned(std::min<int64_t>(1024, std::max<int64_t>(1, (n + 255) / 256)));
}

void launch_scan_nonfinite(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                           int* flag, bool clear, hipStream_t stream) {
  FD_REQUIRE(flag != nullptr, FD_ERR_INVALID_ARG, "internal: no flag word");
  if (clear) {
    hipLaunchKernelGGL(clear_flag_kernel, dim3(1), dim3(1), 0, stream, flag);
    FD_LAUNCH_CHECK();
  }
  hipLaunchKernelGGL(scan_nonfinite_kernel, dim3(stride_grid(N * D)), dim3(256), 0, stream, X,
                     xt == FD_BF16 ? 1 : 0, N, int(D), ldx, flag);
  FD_LAUNCH_CHECK();
}

void launch_poison(const int* flag, float* v, int64_t rows, int64_t cols, int64_t ld,
                   hipStream_t stream) {
  if (v == nullptr || rows * cols == 0) return;
  hipLaunchKernelGGL(poison_f32_kernel, dim3(stride_grid(rows * cols)), dim3(256), 0, stream,
                     flag, v, rows, cols, ld);
  FD_LAUNCH_CHECK();
}

void launch_poison(const int* flag, double* v, int64_t n, hipStream_t stream) {
  if (v == nullptr || n == 0) return;
  hipLaunchKernelGGL(poison_f64_kernel, dim3(stride_grid(n)), dim3(256), 0, stream, flag, v, n);
  FD_LAUNCH_CHECK();
}

void require_finite(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx, int* flag,
                    hipStream_t stream) {
  launch_scan_nonfinite(X, xt, N, D, ldx, flag, true, stream);
  int h = 0;
  FD_HIP_CHECK(hipMemcpyAsync(&h, flag, sizeof(int), hipMemcpyDeviceToHost, stream));
  FD_HIP_CHECK(hipStreamSynchronize(stream));
  FD_REQUIRE(h == 0, FD_ERR_INVALID_ARG, "X holds a NaN or infinite value");
}

// ---------------------------------------------------------------- products

ProductWs carve_product(Arena& a, int64_t Nr, int64_t Nc, int64_t D, int b) {
  ProductWs w;
  const int dp = padded_dim(D);
  w.plan = plan_product(Nr, Nc, dp, b);
  w.rows = carve_pack(a, Nr, dp, ROW_PAD);
  w.cols = carve_pack(a, Nc, dp, COL_PAD);
  w.vp = a.fspan(size_t(w.cols.npad) * w.plan.ncb * 16);
  w.vscale = a.fspan(128);
  w.part = a.fspan(part_rows_bound(w.rows.npad, Nc) * w.plan.ncb * 16);
  w.tmp = a.fspan(size_t(Nr));
  w.flag = a.take<int>(1);
  w.centre = carve_centre(a, Nc);
  return w;
}

// The same regions sized for exactly the plan the call will run (the bound
// above covers every plan up to the given sizes).
static ProductWs carve_product_exact(Arena& a, int64_t Nr, int64_t Nc, int64_t D, int b) {
  ProductWs w;
  const int dp = padded_dim(D);
  w.plan = plan_product(Nr, Nc, dp, b);
  w.rows = carve_pack(a, Nr, dp, ROW_PAD);
  w.cols = carve_pack(a, Nc, dp, COL_PAD);
  w.vp = a.fspan(size_t(w.cols.npad) * w.plan.ncb * 16);
  w.vscale = a.fspan(128);
  const KVPlan rp = plan_rowsum(Nr, Nc, dp);
  const size_t part_prod = size_t(w.plan.nsplit) * w.rows.npad * w.plan.ncb * 16;
  const size_t part_row = size_t(rp.nsplit) * w.rows.npad;
  w.part = a.fspan(b == 1 ? part_row : part_prod);
  w.tmp = a.fspan(size_t(Nr));
  w.flag = a.take<int>(1);
  w.centre = carve_centre(a, Nc);
  return w;
}

// Scratch of the allocation-free product: one array per device, held until
// the process ends.  Host code never passes the array's name to a kernel or a
// copy (on the host it is a stand-in, not a device address); it uses the
// device address that hipGetSymbolAddress returns, looked up once per device
// with that device current.
constexpr size_t SCRATCH_BYTES = size_t(256) << 20;
static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

static char* scratch_on_current_device() {
  static std::mutex mu;
  static std::vector<char*> ptrs;
  int dev = -1;
  FD_HIP_CHECK(hipGetDevice(&dev));
  FD_REQUIRE(dev >= 0, FD_ERR_HIP, "no current device");
  std::lock_guard<std::mutex> lock(mu);
  if (size_t(dev) >= ptrs.size()) ptrs.resize(size_t(dev) + 1, nullptr);
  if (ptrs[size_t(dev)] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    FD_REQUIRE(e == hipSuccess && p != nullptr, FD_ERR_HIP,
               std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    FD_REQUIRE((reinterpret_cast<uintptr_t>(p) & 255) == 0, FD_ERR_HIP,
               "scratch array is not 256-byte aligned");
    ptrs[size_t(dev)] = static_cast<char*>(p);
  }
  return ptrs[size_t(dev)];
}

// Every plan has nsplit <= max(ceil(2048 / row blocks), ceil(column tiles /
// SPLIT_SPAN_TILES)), so the partial buffers of any problem with at most npad
// rows and nc columns fit in this many row slots.
size_t part_rows_bound(int64_t npad, int64_t nc) {
  return size_t(2048) * ROW_PAD + size_t(npad) * size_t(1 + ceil_div(ceil_div(nc, TILE), SPLIT_SPAN_TILES));
}

PointPack pack_view(const PointPack& big, int64_t n, int64_t pad) {
  PointPack p = big;
  p.n = n;
  p.npad = round_up(n, pad);
  return p;
}

DegreeWs degree_view(const DegreeWs& big, int64_t n) {
  DegreeWs w = big;
  w.rows = pack_view(big.rows, n, ROW_PAD);
  w.cols = pack_view(big.cols, n, COL_PAD);
  w.plan = plan_rowsum(n, n, big.rows.dp);
  return w;
}

ProductWs product_view(const ProductWs& big, const PointPack& rows, const PointPack& cols,
                       int width) {
  ProductWs w = big;
  w.rows = rows;
  w.cols = cols;
  w.plan = plan_product(rows.n, cols.n, rows.dp, width);
  return w;
}

void product_apply(ProductWs& w, const float* sl, const float* sr, const float* V, int64_t ldv,
                   int b, float* Y, int64_t ldy, bool diag, hipStream_t stream) {
  if (b == 1) {
    // one right-hand side: weighted row sums K (sr v) on the vector ALUs (no
    // matrix-core contraction padded to 16 columns), then the row scale
    launch_pack_wv(V, ldv, sr, w.cols.n, w.cols.npad, w.vp, stream);
    const KVPlan rp = plan_rowsum(w.rows.n, w.cols.n, w.rows.dp);
    check_span(w.tmp, size_t(w.rows.n), "single-column row sums");
    launch_rowsum(rp, w.rows, w.cols, w.vp, diag, w.tmp.p, w.part, stream);
    launch_scale_rows(w.tmp.p, sl, w.rows.n, Y, ldy, stream);
    return;
  }
  launch_pack_v_for(w.rows, V, w.cols.n, b, ldv, sr, w.plan.ncb, w.cols.npad, w.vp, w.vscale,
                    stream);
  launch_product(w.plan, w.rows, w.cols, w.vp, w.vscale, diag, sl, Y, ldy, b, w.part, stream);
}

// ---------------------------------------------------------------- degree

DegreeWs carve_degree(Arena& a, int64_t N, int64_t D) {
  DegreeWs w;
  const int dp = padded_dim(D);
  w.plan = plan_rowsum(N, N, dp);
  w.rows = carve_pack(a, N, dp, ROW_PAD);
  w.cols = carve_pack(a, N, dp, COL_PAD);
  w.wp = a.fspan(size_t(w.cols.npad) * 16);  // one float4 per lane per 16-point tile
  w.q = a.take<float>(size_t(N));
  w.t = a.take<float>(size_t(N));
  w.w = a.take<float>(size_t(N));
  w.part = a.fspan(std::max(part_rows_bound(w.rows.npad, N), sym_part_rows(w.rows.npad, SYM_NIB)));
  w.colfix = a.take<unsigned long long>(size_t(w.rows.npad));
  w.flag = a.take<int>(1);
  w.centre = carve_centre(a, N);
  return w;
}

void degree_run(DegreeWs& w, const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                double beta, double alpha, float* q, float* d, float* s, double* s_off,
                bool pack, hipStream_t stream) {
  if (pack) {
    launch_centre(X, xt, N, D, ldx, w.centre, stream);
    launch_pack_points(X, xt, N, D, ldx, beta, true, w.rows, &w.centre, stream);
    launch_pack_points(X, xt, N, D, ldx, beta, false, w.cols, &w.centre, stream);
  }
  float* qq = q != nullptr ? q : w.q;
  if (rowsum_sym_applies(w.rows, w.cols, true, w.colfix)) {
    // symmetric row sums with the epilogues fused into their reductions; the
    // first reduction leaves the column-sum words zeroed for the second pass
    const SymPass p1 = launch_rowsum_sym_pass(w.plan, w.rows, w.cols, FSpan{}, w.part, w.colfix,
                                              true, stream);
    launch_degree_reduce_q(p1, w.rows, w.cols, w.part, w.colfix, qq, alpha,
                           alpha == 0.0 ? FSpan{} : w.wp, stream);
    if (s_off != nullptr) launch_sum_minus_n(qq, N, s_off, stream);
    if (alpha == 0.0) {
      launch_degree_finish(qq, qq, N, 0.0, d, s, stream);
      return;
    }
    const SymPass p2 = launch_rowsum_sym_pass(w.plan, w.rows, w.cols, w.wp, w.part, w.colfix,
                                              false, stream);
    launch_degree_reduce_ds(p2, w.rows, w.part, w.colfix, qq, alpha, d, s, stream);
    return;
  }
  launch_rowsum(w.plan, w.rows, w.cols, FSpan{}, true, qq, w.part, stream, w.colfix);
  if (s_off != nullptr) launch_sum_minus_n(qq, N, s_off, stream);
  if (alpha == 0.0) {
    launch_degree_finish(qq, qq, N, 0.0, d, s, stream);
    return;
  }
  launch_pow_neg(qq, N, alpha, w.w, stream);
  launch_pack_w(w.w, N, w.cols.npad, w.wp, stream);
  launch_rowsum(w.plan, w.rows, w.cols, w.wp, true, w.t, w.part, stream, w.colfix);
  launch_degree_finish(qq, w.t, N, alpha, d, s, stream);
}

DegreeWs carve_degree_dyadic(Arena& a, int64_t N, int64_t D) {
  DegreeWs w = carve_degree(a, N, D);
  w.sq_part = a.fspan(sym_part_rows(w.rows.npad, SYM_NIB));
  w.sq_colfix = a.take<unsigned long long>(size_t(w.rows.npad));
  return w;
}

void degree_run_dyadic(DegreeWs& w, const void* X, fd_dtype xt, int64_t N, int64_t D,
                       int64_t ldx, double beta0, int nb, double alpha, float* q, float* d,
                       float* s, double* s_off, hipStream_t stream) {
  auto at = [N](float* v, int l) { return v != nullptr ? v + int64_t(l) * N : nullptr; };
  auto beta_of = [beta0](int l) { return std::ldexp(beta0, l); };
  launch_centre(X, xt, N, D, ldx, w.centre, stream);
  launch_pack_points(X, xt, N, D, ldx, beta_of(0), true, w.rows, &w.centre, stream);
  launch_pack_points(X, xt, N, D, ldx, beta_of(0), false, w.cols, &w.centre, stream);
  if (alpha == 0.0 || !rowsum_sym_applies(w.rows, w.cols, true, w.colfix)) {
    // no weighted pass to carry the squares (alpha = 0), or not the symmetric
    // path: fd_degree's passes, level by level
    for (int l = 0; l < nb; ++l)
      degree_run(w, X, xt, N, D, ldx, beta_of(l), alpha, at(q, l), at(d, l), at(s, l),
                 s_off != nullptr ? s_off + l : nullptr, l > 0, stream);
    return;
  }
  // q of the current level and of the next, in the caller's arrays or in two
  // workspace vectors used in turn
  auto q_of = [&](int l) { return q != nullptr ? q + int64_t(l) * N : (l % 2 ? w.w : w.q); };
  const SymPass p1 = launch_rowsum_sym_pass(w.plan, w.rows, w.cols, FSpan{}, w.part, w.colfix,
                                            true, stream);
  launch_degree_reduce_q(p1, w.rows, w.cols, w.part, w.colfix, q_of(0), alpha, w.wp, stream);
  if (s_off != nullptr) launch_sum_minus_n(q_of(0), N, s_off, stream);
  launch_zero_u64(w.sq_colfix, w.rows.npad, stream);
  for (int l = 0; l < nb; ++l) {
    if (l > 0) {
      launch_pack_points(X, xt, N, D, ldx, beta_of(l), true, w.rows, &w.centre, stream);
      launch_pack_points(X, xt, N, D, ldx, beta_of(l), false, w.cols, &w.centre, stream);
    }
    if (l + 1 == nb) {
      const SymPass p2 = launch_rowsum_sym_pass(w.plan, w.rows, w.cols, w.wp, w.part, w.colfix,
                                                false, stream);
      launch_degree_reduce_ds(p2, w.rows, w.part, w.colfix, q_of(l), alpha, at(d, l), at(s, l),
                              stream);
      break;
    }
    // weighted pass of level l with the squared sums: t_l and q_{l+1}
    const SymPass p2 = launch_rowsum_sym_pass(w.plan, w.rows, w.cols, w.wp, w.part, w.colfix,
                                              false, stream, w.sq_part, w.sq_colfix);
    launch_degree_reduce_dsq(p2, w.rows, w.cols, w.part, w.colfix, q_of(l), alpha, at(d, l),
                             at(s, l), w.sq_part, w.sq_colfix, q_of(l + 1), w.wp, stream);
    if (s_off != nullptr) launch_sum_minus_n(q_of(l + 1), N, s_off + l + 1, stream);
  }
}

}  // namespace fd

using namespace fd;

extern "C" {

const char* fd_last_error(void) { return get_error(); }

const char* fd_status_string(fd_status s) {
  switch (s) {
    case FD_OK: return "FD_OK";
    case FD_ERR_INVALID_ARG: return "FD_ERR_INVALID_ARG";
    case FD_ERR_UNSUPPORTED: return "FD_ERR_UNSUPPORTED";
    case FD_ERR_WORKSPACE: return "FD_ERR_WORKSPACE";
    case FD_ERR_HIP: return "FD_ERR_HIP";
    case FD_ERR_NOT_CONVERGED: return "FD_ERR_NOT_CONVERGED";
    case FD_ERR_PERRON_WALL: return "FD_ERR_PERRON_WALL";
  }
  return "FD_UNKNOWN_STATUS";
}

void fd_lanczos_default_opts(fd_lanczos_opts* opts) {
  if (opts == nullptr) return;
  opts->tol = 1e-5;
  opts->max_restarts = 200;
  opts->max_basis_blocks = 0;
  opts->keep = -1;
  opts->max_matvecs = 0;
  opts->verbose = 0;
  opts->seed = 0x5eed;
}

size_t fd_workspace_size(fd_op op, int64_t Nr, int64_t Nc, int64_t D, int64_t b, int64_t k,
                         const fd_lanczos_opts* opts) {
  size_t out = 0;
  fd_status st = guarded([&] {
    Arena a;
    a.measuring = true;
    FD_REQUIRE(Nr >= 1 && Nr <= MAX_POINTS && D >= 1 && D <= MAX_D, FD_ERR_INVALID_ARG, "size");
    switch (op) {
      case FD_OP_KERNEL_MATMUL:
        FD_REQUIRE(Nc >= 1 && Nc <= MAX_POINTS && b >= 1 && b <= MAX_B, FD_ERR_INVALID_ARG, "size");
        carve_product(a, Nr, Nc, D, int(b));
        break;
      case FD_OP_DEGREE:
        carve_degree(a, Nr, D);
        break;
      case FD_OP_DEGREE_DYADIC:
        carve_degree_dyadic(a, Nr, D);
        break;
      case FD_OP_BLOCK_LANCZOS: {
        fd_lanczos_opts o;
        fd_lanczos_default_opts(&o);
        if (opts != nullptr) o = *opts;
        FD_REQUIRE(b >= 1 && b <= MAX_B && k >= 1 && k <= Nr, FD_ERR_INVALID_ARG, "size");
        carve_solver(a, Nr, D, int(b), int(k), o);
        break;
      }
      case FD_OP_CONTINUATION: {
        fd_lanczos_opts o;
        fd_lanczos_default_opts(&o);
        if (opts != nullptr) o = *opts;
        FD_REQUIRE(b >= 1 && b <= MAX_B && k >= 1 && k <= 64 && k <= Nr && Nc >= 1,
                   FD_ERR_INVALID_ARG, "size");
        carve_continuation_ws(a, Nr, Nc, D, int(b), int(k), o);
        break;
      }
      case FD_OP_BETA_FLOW: {
        fd_lanczos_opts o;
        fd_lanczos_default_opts(&o);
        if (opts != nullptr) o = *opts;
        FD_REQUIRE(b >= 1 && b <= MAX_B && k >= 2 && k <= Nr, FD_ERR_INVALID_ARG, "size");
        carve_flow_ws(a, Nr, D, int(b), int(k), o);
        break;
      }
      default:
        throw Error{FD_ERR_INVALID_ARG, "unknown op"};
    }
    out = a.used;
  });
  return st == FD_OK ? out : 0;
}

fd_status fd_kernel_matmul(const void* Xr, int64_t Nr, const void* Xc, int64_t Nc, int64_t D,
                           int64_t ldx, fd_dtype xt, float beta, const float* sl, const float* sr,
                           const float* V, int64_t b, int64_t ldv, float* Y, int64_t ldy,
                           void* ws, size_t ws_bytes, void* stream) {
  return guarded([&] {
    check_points(Xr, xt, Nr, D, ldx, "Xr");
    check_points(Xc, xt, Nc, D, ldx, "Xc");
    FD_REQUIRE(std::isfinite(beta) && beta >= 0.f, FD_ERR_INVALID_ARG, "beta must be finite and >= 0");
    FD_REQUIRE(V != nullptr && Y != nullptr, FD_ERR_INVALID_ARG, "V and Y must not be NULL");
    FD_REQUIRE(b >= 1 && b <= MAX_B, FD_ERR_INVALID_ARG, "b must be in [1, 64]");
    FD_REQUIRE(ldv >= b && ldy >= b, FD_ERR_INVALID_ARG, "ldv and ldy must be >= b");
    Arena m;
    m.measuring = true;
    carve_product(m, Nr, Nc, D, int(b));
    check_workspace(ws, ws_bytes, m.used);
    Arena a;
    a.base = static_cast<char*>(ws);
    a.cap = ws_bytes;
    ProductWs w = carve_product(a, Nr, Nc, D, int(b));
    hipStream_t st = static_cast<hipStream_t>(stream);
    launch_scan_nonfinite(Xr, xt, Nr, D, ldx, w.flag, true, st);
    if (Xc != Xr) launch_scan_nonfinite(Xc, xt, Nc, D, ldx, w.flag, false, st);
    // one centre for both sets: the column set's mean, the radius over both
    launch_centre(Xc, xt, Nc, D, ldx, w.centre, st);
    if (Xr != Xc || Nr > Nc) launch_radius_more(Xr, xt, Nr, D, ldx, w.centre, st);
    launch_pack_points(Xr, xt, Nr, D, ldx, beta, true, w.rows, &w.centre, st);
    launch_pack_points(Xc, xt, Nc, D, ldx, beta, false, w.cols, &w.centre, st);
    // same base pointer and ldx: index i names the same point in both sets
    const bool diag = (Xr == Xc);
    product_apply(w, sl, sr, V, ldv, int(b), Y, ldy, diag, st);
    launch_range_check(xt, w.centre, beta, w.flag, st);
    launch_poison(w.flag, Y, Nr, b, ldy, st);
  });
}

fd_status fd_kernel_matmul_noalloc(const void* Xr, int64_t Nr, const void* Xc, int64_t Nc,
                                   int64_t D, int64_t ldx, fd_dtype xt, float beta,
                                   const float* sl, const float* sr, const float* V, int64_t b,
                                   int64_t ldv, float* Y, int64_t ldy, void* stream) {
  return guarded([&] {
    check_points(Xr, xt, Nr, D, ldx, "Xr");
    check_points(Xc, xt, Nc, D, ldx, "Xc");
    FD_REQUIRE(std::isfinite(beta) && beta >= 0.f, FD_ERR_INVALID_ARG, "beta must be finite and >= 0");
    FD_REQUIRE(V != nullptr && Y != nullptr, FD_ERR_INVALID_ARG, "V and Y must not be NULL");
    FD_REQUIRE(b >= 1 && b <= MAX_B, FD_ERR_INVALID_ARG, "b must be in [1, 64]");
    FD_REQUIRE(ldv >= b && ldy >= b, FD_ERR_INVALID_ARG, "ldv and ldy must be >= b");
    Arena m;
    m.measuring = true;
    carve_product_exact(m, Nr, Nc, D, int(b));
    FD_REQUIRE(m.used <= SCRATCH_BYTES, FD_ERR_WORKSPACE,
               "problem too large for the built-in scratch: needs " + std::to_string(m.used) +
                   " bytes, the scratch holds " + std::to_string(SCRATCH_BYTES) +
                   " (use fd_kernel_matmul with a workspace)");
    Arena a;
    a.base = scratch_on_current_device();
    a.cap = SCRATCH_BYTES;
    ProductWs w = carve_product_exact(a, Nr, Nc, D, int(b));
    hipStream_t st = static_cast<hipStream_t>(stream);
    launch_scan_nonfinite(Xr, xt, Nr, D, ldx, w.flag, true, st);
    if (Xc != Xr) launch_scan_nonfinite(Xc, xt, Nc, D, ldx, w.flag, false, st);
    // one centre for both sets: the column set's mean, the radius over both
    launch_centre(Xc, xt, Nc, D, ldx, w.centre, st);
    if (Xr != Xc || Nr > Nc) launch_radius_more(Xr, xt, Nr, D, ldx, w.centre, st);
    launch_pack_points(Xr, xt, Nr, D, ldx, beta, true, w.rows, &w.centre, st);
    launch_pack_points(Xc, xt, Nc, D, ldx, beta, false, w.cols, &w.centre, st);
    const bool diag = (Xr == Xc);
    product_apply(w, sl, sr, V, ldv, int(b), Y, ldy, diag, st);
    launch_range_check(xt, w.centre, beta, w.flag, st);
    launch_poison(w.flag, Y, Nr, b, ldy, st);
  });
}

size_t fd_kernel_matmul_noalloc_limit(void) { return SCRATCH_BYTES; }

fd_status fd_degree(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx, float beta,
                    float alpha, float* q, float* d, float* s, double* s_off, void* ws,
                    size_t ws_bytes, void* stream) {
  return guarded([&] {
    check_points(X, xt, N, D, ldx, "X");
    FD_REQUIRE(std::isfinite(beta) && beta > 0.f, FD_ERR_INVALID_ARG, "beta must be finite and > 0");
    FD_REQUIRE(alpha >= 0.f && alpha <= 1.f, FD_ERR_INVALID_ARG, "alpha must be in [0, 1]");
    Arena m;
    m.measuring = true;
    carve_degree(m, N, D);
    check_workspace(ws, ws_bytes, m.used);
    Arena a;
    a.base = static_cast<char*>(ws);
    a.cap = ws_bytes;
    DegreeWs w = carve_degree(a, N, D);
    hipStream_t st = static_cast<hipStream_t>(stream);
    launch_scan_nonfinite(X, xt, N, D, ldx, w.flag, true, st);
    degree_run(w, X, xt, N, D, ldx, beta, alpha, q, d, s, s_off, true, st);
    launch_range_check(xt, w.centre, beta, w.flag, st);
    for (float* v : {q, d, s}) launch_poison(w.flag, v, N, 1, 1, st);
    launch_poison(w.flag, s_off, 1, st);
  });
}

fd_status fd_degree_dyadic(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                           float beta0, int32_t nbeta, float alpha, float* q, float* d, float* s,
                           double* s_off, void* ws, size_t ws_bytes, void* stream) {
  return guarded([&] {
    check_points(X, xt, N, D, ldx, "X");
    FD_REQUIRE(nbeta >= 1 && nbeta <= 32, FD_ERR_INVALID_ARG, "nbeta must be in [1, 32]");
    FD_REQUIRE(std::isfinite(beta0) && beta0 > 0.f &&
                   std::isfinite(std::ldexp(double(beta0), nbeta - 1)) &&
                   std::ldexp(double(beta0), nbeta - 1) <= double(FLT_MAX),
               FD_ERR_INVALID_ARG, "beta0 must be > 0 with beta0 2^(nbeta-1) finite");
    FD_REQUIRE(alpha >= 0.f && alpha <= 1.f, FD_ERR_INVALID_ARG, "alpha must be in [0, 1]");
    Arena m;
    m.measuring = true;
    carve_degree_dyadic(m, N, D);
    check_workspace(ws, ws_bytes, m.used);
    Arena a;
    a.base = static_cast<char*>(ws);
    a.cap = ws_bytes;
    DegreeWs w = carve_degree_dyadic(a, N, D);
    hipStream_t st = static_cast<hipStream_t>(stream);
    launch_scan_nonfinite(X, xt, N, D, ldx, w.flag, true, st);
    degree_run_dyadic(w, X, xt, N, D, ldx, beta0, int(nbeta), alpha, q, d, s, s_off, st);
    // the largest bandwidth decides (every level's outputs are poisoned)
    launch_range_check(xt, w.centre, std::ldexp(double(beta0), nbeta - 1), w.flag, st);
    for (float* v : {q, d, s}) launch_poison(w.flag, v, int64_t(nbeta) * N, 1, 1, st);
    launch_poison(w.flag, s_off, nbeta, st);
  });
}

}  // extern "C"
