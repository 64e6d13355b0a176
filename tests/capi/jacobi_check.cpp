// Internal check of the dense symmetric eigensolve behind the eigensolver's
// Rayleigh-Ritz step (fd::jacobi_eig in libflashdiff.so) on matrices whose
// diagonal holds NaN, on the one-workgroup path (m <= 192) and the block path.
// Both must finish, and the eigenvalues must come back with every number
// sorted descending before the NaNs: the sort ranks the diagonal in a strict
// total order, so its gather of eigenvector columns stays a permutation (a
// rank order with plain comparisons left rank slots unwritten on a NaN
// diagonal and gathered from an index out of range).
// Prints one line per size; exit status 0 when every check holds.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <random>
#include <vector>

#include "fd_linalg.hpp"

namespace {

bool check(int m, unsigned seed) {
  std::mt19937_64 g(seed);
  std::normal_distribution<double> nd;
  std::vector<double> A(size_t(m) * m);
  for (int i = 0; i < m; ++i)
    for (int j = i; j < m; ++j) {
      const double v = i == j ? 1.0 + 0.1 * nd(g) : 0.05 * nd(g);
      A[size_t(i) * m + j] = A[size_t(j) * m + i] = v;
    }
  A[size_t(7) * m + 7] = NAN;
  A[size_t(m - 3) * m + m - 3] = NAN;
  const size_t nlog = fd::jacobi_log_doubles(m);
  double *dA = nullptr, *dA2 = nullptr, *dV = nullptr, *dS = nullptr, *dth = nullptr,
         *dn = nullptr, *dlog = nullptr;
  int* dst = nullptr;
  const size_t mm = size_t(m) * m * sizeof(double);
  if (hipMalloc(&dA, mm) != hipSuccess || hipMalloc(&dA2, mm) != hipSuccess ||
      hipMalloc(&dV, mm) != hipSuccess || hipMalloc(&dS, mm) != hipSuccess ||
      hipMalloc(&dth, m * sizeof(double)) != hipSuccess ||
      hipMalloc(&dn, 2 * sizeof(double)) != hipSuccess ||
      hipMalloc(&dlog, nlog * sizeof(double)) != hipSuccess ||
      hipMalloc(&dst, 2 * sizeof(int)) != hipSuccess) {
    std::printf("m %d: allocation failed\n", m);
    return false;
  }
  hipStream_t st = nullptr;
  bool ok = hipMemcpy(dA, A.data(), mm, hipMemcpyHostToDevice) == hipSuccess;
  int sweeps = -1;
  try {
    sweeps = fd::jacobi_eig(dA, dA2, m, m, dV, dth, dS, m, dn, fd::FSpanD{dlog, nlog}, dst, st);
  } catch (const fd::Error& e) {
    std::printf("m %d: jacobi_eig raised: %s\n", m, e.msg.c_str());
    ok = false;
  }
  std::vector<double> th(m);
  ok = ok && hipDeviceSynchronize() == hipSuccess &&
       hipMemcpy(th.data(), dth, m * sizeof(double), hipMemcpyDeviceToHost) == hipSuccess;
  int first_nan = m;
  for (int i = 0; i < m; ++i)
    if (std::isnan(th[i])) {
      first_nan = i;
      break;
    }
  bool sorted = true;
  for (int i = 0; i < m; ++i) {
    if (i >= first_nan && !std::isnan(th[i])) sorted = false;
    if (i + 1 < first_nan && th[i] < th[i + 1]) sorted = false;
  }
  std::printf("m %d: %s, sweeps %d, %d numbers then %d NaN, order %s\n", m,
              ok ? "finished" : "FAILED", sweeps, first_nan, m - first_nan,
              sorted ? "ok" : "WRONG");
  for (void* p : {(void*)dA, (void*)dA2, (void*)dV, (void*)dS, (void*)dth, (void*)dn,
                  (void*)dlog, (void*)dst})
    (void)hipFree(p);
  return ok && sorted;
}

}  // namespace

int main() {
  bool all = true;
  for (int m : {100, 300}) all = check(m, 17u + unsigned(m)) && all;
  return all ? 0 : 1;
}
