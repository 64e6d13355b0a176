// Internal check of the dense helpers of the eigensolver's
// reorthogonalisation and restarts in libflashdiff.so against the host.
// The tall-skinny products (fd::gemm_tn, fd::gemm_nn) are compared with
// float64 sums on the host on shapes that take every load path: vector and
// scalar loads, one to four 16-column blocks per wave (partly used ones too),
// one and several column tiles, 16 to 64 rows per wave, ragged row counts
// (not a multiple of the 64 rows a workgroup takes per step), offset and odd
// leading dimensions, and N from 1 to 2^18 + 3 rows.
//   gemm_tn: C = A^T B in float64 from float32 inputs.  Every product of two
//     float32 values is exact in float64, so C differs from the host's
//     sequential float64 sum only by the two summation orders: the bound is
//     2 N eps sum |a b|.
//   gemm_nn: Z = beta Z + alpha Q C in float32 (sums in the float32 matrix
//     unit); against the float64 value the bound is
//     (ma + 2) 2^-24 (|beta z| + |alpha| sum |q c|).
//   chol_rinv: G = R^T R of a Gram matrix G = Y^T Y and Rinv = R^-1 (float32).
//     Checked: Rinv is upper triangular and Rinv^T G Rinv = I on the
//     unflagged columns to float32 rounding (1e-5); no flags on a full-rank
//     G; on a G whose listed columns repeat the column before them (and one
//     column is zero) exactly those columns are flagged and their rows of
//     Rinv are unit rows.
// Prints one line per case; exit status 0 when every check holds.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "fd_linalg.hpp"

namespace {

float val(uint64_t i) { return float((i * 2654435761ull) % 1000003ull) * 1e-6f - 0.5f; }

template <class T>
T* dev(const std::vector<T>& h) {
  T* p = nullptr;
  if (hipMalloc(&p, h.size() * sizeof(T)) != hipSuccess) return nullptr;
  if (hipMemcpy(p, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice) != hipSuccess) return nullptr;
  return p;
}

struct TnCase {
  int ma;
  int64_t lda;
  int nb;
  int64_t ldb, N;
  int aoff, boff;
  bool full;  // every entry against the host (else a sample of 1 in 97)
};

bool check_tn(const TnCase& c) {
  const size_t na = size_t(c.N - 1) * c.lda + c.ma + c.aoff;
  const size_t nbv = size_t(c.N - 1) * c.ldb + c.nb + c.boff;
  std::vector<float> ha(na), hb(nbv);
  for (size_t i = 0; i < na; ++i) ha[i] = val(i);
  for (size_t i = 0; i < nbv; ++i) hb[i] = val(i + 77777);
  float* A = dev(ha);
  float* B = dev(hb);
  const size_t np = size_t(fd::gemm_tn_chunks(c.N)) * c.ma * c.nb;
  double *C = nullptr, *part = nullptr;
  float* C32 = nullptr;
  bool ok = A && B && hipMalloc(&C, size_t(c.ma) * c.nb * 8) == hipSuccess &&
            hipMalloc(&C32, size_t(c.ma) * c.nb * 4) == hipSuccess &&
            hipMalloc(&part, np * 8) == hipSuccess;
  std::vector<double> hc(size_t(c.ma) * c.nb);
  std::vector<float> hc32(hc.size());
  if (ok) {
    try {
      fd::gemm_tn(A + c.aoff, c.lda, c.ma, B + c.boff, c.ldb, c.nb, c.N, fd::FSpanD{part, np}, C,
                  C32, nullptr);
    } catch (const fd::Error& e) {
      std::printf("gemm_tn raised: %s\n", e.msg.c_str());
      ok = false;
    }
    ok = ok && hipDeviceSynchronize() == hipSuccess &&
         hipMemcpy(hc.data(), C, hc.size() * 8, hipMemcpyDeviceToHost) == hipSuccess &&
         hipMemcpy(hc32.data(), C32, hc32.size() * 4, hipMemcpyDeviceToHost) == hipSuccess;
  }
  double worst = 0.0;
  long checked = 0;
  bool copy_ok = true;
  for (int l = 0; ok && l < c.ma; ++l)
    for (int j = 0; j < c.nb; ++j) {
      if (hc32[size_t(l) * c.nb + j] != float(hc[size_t(l) * c.nb + j])) copy_ok = false;
      if (!c.full && (l * 131 + j * 7) % 97 != 0) continue;
      double s = 0.0, sa = 0.0;
      for (int64_t r = 0; r < c.N; ++r) {
        const double p = double(ha[c.aoff + r * c.lda + l]) * double(hb[c.boff + r * c.ldb + j]);
        s += p;
        sa += std::fabs(p);
      }
      const double e = std::fabs(hc[size_t(l) * c.nb + j] - s) / (sa > 0.0 ? sa : 1.0);
      if (!(e <= worst)) worst = e;  // a NaN stays the worst
      ++checked;
    }
  const double tol = 2.0 * double(c.N) * 1.1102230246251565e-16;
  const bool pass = ok && copy_ok && worst <= tol;
  std::printf("gemm_tn ma %4d lda %4lld nb %2d ldb %4lld N %6lld offsets %d/%d: %ld checked, "
              "max err / sum|ab| %.2e (bound %.1e), float32 copy %s: %s\n",
              c.ma, (long long)c.lda, c.nb, (long long)c.ldb, (long long)c.N, c.aoff, c.boff, checked,
              worst, tol, copy_ok ? "ok" : "WRONG", pass ? "ok" : "FAILED");
  for (void* p : {(void*)A, (void*)B, (void*)C, (void*)C32, (void*)part}) (void)hipFree(p);
  return pass;
}

struct NnCase {
  int ma;
  int64_t ldq;
  int nb;
  int64_t ldz, N;
  float alpha, beta;
  int row_step = 1;  // rows checked against the host: every row_step-th and the last
};

bool check_nn(const NnCase& c) {
  const size_t nq = size_t(c.N - 1) * c.ldq + c.ma, nz = size_t(c.N - 1) * c.ldz + c.nb;
  std::vector<float> hq(nq), hcm(size_t(c.ma) * c.nb), hz(nz);
  for (size_t i = 0; i < nq; ++i) hq[i] = val(i + 3);
  for (size_t i = 0; i < hcm.size(); ++i) hcm[i] = val(i + 999331);
  for (size_t i = 0; i < nz; ++i) hz[i] = val(i + 4242);
  float* Q = dev(hq);
  float* Cm = dev(hcm);
  float* Z = dev(hz);
  bool ok = Q && Cm && Z;
  std::vector<float> out(nz);
  if (ok) {
    try {
      fd::gemm_nn(Q, c.ldq, c.ma, Cm, c.nb, Z, c.ldz, c.N, c.alpha, c.beta, nullptr);
    } catch (const fd::Error& e) {
      std::printf("gemm_nn raised: %s\n", e.msg.c_str());
      ok = false;
    }
    ok = ok && hipDeviceSynchronize() == hipSuccess &&
         hipMemcpy(out.data(), Z, nz * 4, hipMemcpyDeviceToHost) == hipSuccess;
  }
  double worst = 0.0;
  bool untouched = true;
  for (int64_t r = 0; ok && r < c.N; r = (r + c.row_step < c.N || r == c.N - 1) ? r + c.row_step : c.N - 1) {
    for (int j = 0; j < c.nb; ++j) {
      double s = 0.0, sa = 0.0;
      for (int l = 0; l < c.ma; ++l) {
        const double p = double(hq[r * c.ldq + l]) * double(hcm[size_t(l) * c.nb + j]);
        s += p;
        sa += std::fabs(p);
      }
      const double z0 = hz[r * c.ldz + j];
      const double ref = double(c.beta) * z0 + double(c.alpha) * s;
      const double scale = std::fabs(double(c.beta) * z0) + std::fabs(double(c.alpha)) * sa;
      const double e = std::fabs(double(out[r * c.ldz + j]) - ref) /
                       ((c.ma + 2) * 5.960464477539063e-08 * (scale > 0.0 ? scale : 1.0));
      if (!(e <= worst)) worst = e;
    }
    // the columns between nb and ldz are not written
    for (int64_t j = c.nb; r + 1 < c.N && j < c.ldz; ++j)
      if (out[r * c.ldz + j] != hz[r * c.ldz + j]) untouched = false;
  }
  const bool pass = ok && untouched && worst <= 1.0;
  std::printf("gemm_nn ma %4d ldq %4lld nb %2d ldz %4lld N %6lld alpha %g beta %g (rows 1 in %d): "
              "max err / bound %.2f, columns past nb %s: %s\n",
              c.ma, (long long)c.ldq, c.nb, (long long)c.ldz, (long long)c.N, c.alpha, c.beta,
              c.row_step, worst, untouched ? "untouched" : "WRITTEN", pass ? "ok" : "FAILED");
  for (void* p : {(void*)Q, (void*)Cm, (void*)Z}) (void)hipFree(p);
  return pass;
}

// Gram matrix Y^T Y of an nr x b matrix Y (float64); columns listed in dup
// copy the column before them, column `zero` (if >= 0) is 0
std::vector<double> gram(int b, int nr, const std::vector<int>& dup, int zero, unsigned seed) {
  // normal entries (the linear index hash of the product checks would give
  // a Gram matrix of rank about 2)
  std::mt19937_64 g(seed);
  std::normal_distribution<double> nd;
  std::vector<double> Y(size_t(nr) * b);
  for (double& y : Y) y = nd(g);
  for (int j : dup)
    for (int i = 0; i < nr; ++i) Y[size_t(i) * b + j] = Y[size_t(i) * b + j - 1];
  if (zero >= 0)
    for (int i = 0; i < nr; ++i) Y[size_t(i) * b + zero] = 0.0;
  std::vector<double> G(size_t(b) * b, 0.0);
  for (int i = 0; i < nr; ++i)
    for (int p = 0; p < b; ++p)
      for (int q = 0; q < b; ++q) G[size_t(p) * b + q] += Y[size_t(i) * b + p] * Y[size_t(i) * b + q];
  return G;
}

bool check_chol(int b, const std::vector<int>& dup, int zero) {
  const std::vector<double> G = gram(b, 3 * b + 5, dup, zero, 1234u * b);
  double* dG = dev(G);
  float* dR = nullptr;
  int* dF = nullptr;
  bool ok = dG && hipMalloc(&dR, size_t(b) * b * 4) == hipSuccess &&
            hipMalloc(&dF, size_t(b) * 4) == hipSuccess;
  std::vector<float> Ri(size_t(b) * b);
  std::vector<int> fl(b);
  if (ok) {
    fd::chol_rinv(dG, b, 1e-4, dR, dF, nullptr);
    ok = hipDeviceSynchronize() == hipSuccess &&
         hipMemcpy(Ri.data(), dR, Ri.size() * 4, hipMemcpyDeviceToHost) == hipSuccess &&
         hipMemcpy(fl.data(), dF, fl.size() * 4, hipMemcpyDeviceToHost) == hipSuccess;
  }
  // expected flags
  std::vector<int> want(b, 0);
  for (int j : dup) want[j] = 1;
  if (zero >= 0) want[zero] = 1;
  bool flags_ok = ok;
  for (int j = 0; ok && j < b; ++j) flags_ok = flags_ok && fl[j] == want[j];
  // R from Rinv (float64 inverse of the float32 triangle) would mix two
  // roundings; check Rinv directly: lower part zero, and on the unflagged
  // columns (Rinv^T G Rinv)[p][q] = delta_pq to float32 rounding
  double lower = 0.0, orth = 0.0;
  for (int p = 0; ok && p < b; ++p)
    for (int q = 0; q < p; ++q) lower = std::fmax(lower, std::fabs(double(Ri[size_t(p) * b + q])));
  for (int p = 0; ok && p < b; ++p) {
    if (want[p]) continue;
    for (int q = 0; q < b; ++q) {
      if (want[q]) continue;
      double s = 0.0;
      for (int u = 0; u < b; ++u)
        for (int v = 0; v < b; ++v)
          s += double(Ri[size_t(u) * b + p]) * G[size_t(u) * b + v] * double(Ri[size_t(v) * b + q]);
      orth = std::fmax(orth, std::fabs(s - (p == q ? 1.0 : 0.0)));
    }
  }
  // the unit rows of flagged columns: Rinv row j = e_j
  bool unit_ok = true;
  for (int j = 0; ok && j < b; ++j)
    if (want[j])
      for (int q = 0; q < b; ++q)
        if (q > j && Ri[size_t(j) * b + q] != 0.f) unit_ok = false;
  const bool pass = ok && flags_ok && unit_ok && lower == 0.0 && orth <= 1e-5;
  std::printf("chol_rinv b %2d, %zu repeated + %s zero column: flags %s, unit rows %s, "
              "lower part %.1e, max |Rinv^T G Rinv - I| %.2e: %s\n",
              b, dup.size(), zero >= 0 ? "one" : "no", flags_ok ? "ok" : "WRONG",
              unit_ok ? "ok" : "WRONG", lower, orth, pass ? "ok" : "FAILED");
  for (void* p : {(void*)dG, (void*)dR, (void*)dF}) (void)hipFree(p);
  return pass;
}

}  // namespace

int main() {
  const TnCase tn[] = {
      {1, 1, 1, 1, 1, 0, 0, true},            // one row, one column: scalar loads
      {4, 4, 2, 2, 63, 0, 0, true},           // fewer rows than one workgroup step
      {100, 101, 7, 9, 1001, 0, 0, true},     // odd leading dimensions: scalar loads
      {96, 96, 32, 96, 16421, 0, 32, true},   // a column block of a wider B, ragged N
      {64, 64, 64, 64, 3000, 0, 0, true},     // two column tiles
      {68, 72, 18, 19, 777, 0, 0, true},      // partial tiles in both directions
      {68, 72, 18, 18, 777, 4, 1, true},      // B not 8-byte aligned
      {32, 32, 16, 16, 100000, 0, 0, true},   // one 16-column block per wave
      {200, 204, 33, 36, 4097, 0, 2, true},   // odd nb
      {64, 64, 17, 17, 5000, 0, 0, true},     // two 16-column blocks, the second one column
      {300, 1024, 50, 1024, 70001, 0, 512, false},
      {1024, 1024, 32, 1024, 262147, 0, 992, false},  // the widest basis, 2^18 + 3 rows
  };
  const NnCase nn[] = {
      {1, 1, 1, 1, 5, 1.f, 0.f},          {100, 101, 7, 9, 1001, -1.f, 1.f},
      {64, 64, 32, 64, 3001, -1.f, 1.f},  {96, 1024, 32, 1024, 4099, 1.f, 0.f},
      {256, 256, 64, 64, 2048, 1.f, 0.f}, {68, 72, 20, 24, 777, 0.5f, -2.f},
      // four 16-column blocks, partly used: vector path (48) and scalar path (50)
      {96, 96, 48, 48, 3001, -1.f, 1.f},  {96, 96, 50, 52, 3001, -1.f, 1.f},
      // 32 and 64 rows per wave (N >= 2^17 and 2^18), ragged N
      {96, 128, 32, 128, 131075, -1.f, 1.f, 97}, {64, 64, 64, 64, 131075, 1.f, 0.f, 97},
      {96, 128, 32, 128, 262147, -1.f, 1.f, 97}, {64, 64, 64, 64, 262147, 1.f, 0.f, 97},
      {100, 101, 7, 9, 262147, -1.f, 1.f, 97},
  };
  bool all = true;
  for (const TnCase& c : tn) all = check_tn(c) && all;
  for (const NnCase& c : nn) all = check_nn(c) && all;
  all = check_chol(1, {}, -1) && all;
  all = check_chol(7, {}, -1) && all;
  all = check_chol(32, {}, -1) && all;
  all = check_chol(64, {}, -1) && all;
  all = check_chol(32, {5, 17}, 9) && all;
  all = check_chol(64, {5, 17, 63}, 40) && all;
  std::printf("%s\n", all ? "all ok" : "FAILED");
  return all ? 0 : 1;
}
