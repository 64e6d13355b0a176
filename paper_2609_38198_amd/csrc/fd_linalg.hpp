// Dense helpers of the eigensolver (device side, see linalg.hip).
#pragma once

#include "fd_internal.hpp"

namespace fd {

struct FSpanD {
  double* p = nullptr;
  size_t n = 0;
};

inline void check_span_d(const FSpanD& s, size_t need, const char* what) {
  if (s.p == nullptr || s.n < need)
    throw Error{FD_ERR_WORKSPACE, std::string("internal: region '") + what +
                                      "' smaller than the extent its kernel touches"};
}

inline FSpanD take_d(Arena& a, size_t count) { return FSpanD{a.take<double>(count), count}; }

// Number of row chunks gemm_tn splits N into (its partial buffer holds
// chunks * ma * nb doubles).
int64_t gemm_tn_chunks(int64_t N);

// C (ma x nb, float64 and/or float32 copies, ld nb) = A[0:N, 0:ma]^T B[0:N, 0:nb].
void gemm_tn(const float* A, int64_t lda, int ma, const float* B, int64_t ldb, int nb, int64_t N,
             FSpanD part, double* C, float* C32, hipStream_t stream);
// Z[0:N, 0:nb] = beta Z + alpha Q[0:N, 0:ma] C (C float32 ma x nb, ld nb); nb <= 64.
// Z must not overlap Q.
void gemm_nn(const float* Q, int64_t ldq, int ma, const float* C, int nb, float* Z, int64_t ldz,
             int64_t N, float alpha, float beta, hipStream_t stream);
// Cholesky of G (b x b) with dependent-column flags; Rinv float32 (ld b).
void chol_rinv(const double* G, int b, double rel_tol, float* Rinv, int* flags,
               hipStream_t stream);
// Normal(0, 1) fill of the flagged columns (all columns when flags == NULL).
void fill_normal(float* Z, int64_t ldz, int64_t N, int nb, const int* flags, uint64_t seed,
                 uint64_t stream_id, hipStream_t stream);
// out[c] = ||W[:, c] - theta_c Y[:, c]||_2 for c < nc (Y, W share ld).
void residual_norms(const float* Y, const float* W, int64_t ld, int nc, const double* theta,
                    int64_t N, FSpanD part, double* out, hipStream_t stream);
// Symmetric eigensolve of A (m x m, m <= 1024, overwritten; only its upper
// triangle is read; A2 an m x m scratch with the same ld): theta descending,
// S columns.  Vw: m x m scratch
// (ld m); norms: 2 doubles of
// scratch; log: jacobi_log_doubles(m) doubles (enough for every size up to m;
// the rotation log of the one-workgroup path for m <= 192, the block
// rotations of the block path above) and state: 2 ints of scratch.
// Synchronises the stream once per sweep (once per few sweeps on the
// one-workgroup path).  Returns the number of sweeps run.
size_t jacobi_log_doubles(int m);
int jacobi_eig(double* A, double* A2, int m, int lda, double* Vw, double* theta, double* S,
               int lds, double* norms, FSpanD log, int* state, hipStream_t stream);
void copy_cols(const float* src, int64_t lds, float* dst, int64_t ldd, int64_t N, int nc,
               const float* scale, double power, hipStream_t stream);
void sub_theta(const float* Y, float* W, int64_t ld, int64_t N, int nc, const double* theta,
               hipStream_t stream);
void put_block(double* T, int ldt, const double* C, int m, int c0, int nb, hipStream_t stream);
void set_diag(double* T, int ldt, int mm, const double* theta, int kk, hipStream_t stream);
void narrow(const double* S, int lds, int m, int nc, float* S32, hipStream_t stream);
// L = (3 I - G) / 2 (float32, column chunks of width nc: chunk c0 at L + kk c0
// with ld min(nc, kk - c0)) for a Gram matrix G (kk x kk, ld ldg); dev = max |G - I|.
void loewdin(const double* G, int ldg, int kk, int nc, float* L, double* dev, hipStream_t stream);
void copy_square(const double* src, int lds, double* dst, int ldd, int m, hipStream_t stream);

}  // namespace fd

namespace fd {
void gather_residuals(const float* Q, const float* W, int64_t ld, const double* theta,
                      const int* sel, int nsel, float* Z, int64_t ldz, int64_t N,
                      hipStream_t stream);
void set_identity(float* Q, int64_t ld, int64_t N, int nc, hipStream_t stream);
}  // namespace fd
