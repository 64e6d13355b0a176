// Dense helpers of the block Lanczos eigensolver, all on the device:
//   * tall-skinny products C = A^T B (reduction over N rows, float64 partial
//     sums reduced in a fixed order) and Z = beta Z + alpha Q C,
//   * Cholesky of a small Gram matrix with detection of dependent columns,
//   * refill of such columns from a counter-based normal generator,
//   * residual norms ||W s - theta Q s|| of Ritz pairs,
//   * cyclic Jacobi eigensolver for the small symmetric projected matrix.
// Everything is deterministic: no atomics, fixed reduction orders.
#include <cmath>

#include "fd_linalg.hpp"

namespace fd {

static inline unsigned nblk(int64_t n, int t) { return unsigned((n + t - 1) / t); }

// ------------------------------------------------------------ C = A^T B
// Grid (l tiles of 64, row chunks).  Thread (lg, cg) accumulates a 4 x 4
// block C[l0 + 4 lg + u][4 cg + v] in float64 over its chunk of rows.
__global__ __launch_bounds__(256) void gemm_tn_partial_kernel(
    const float* __restrict__ A, int64_t lda, int ma, const float* __restrict__ B, int64_t ldb,
    int nb, int64_t N, int64_t rows_per_chunk, double* __restrict__ part) {
  const int lg = threadIdx.x >> 4, cg = threadIdx.x & 15;
  const int l0 = blockIdx.x * 64 + 4 * lg;
  const int c0 = 4 * cg;
  const int64_t chunk = blockIdx.y;
  const int64_t r0 = chunk * rows_per_chunk;
  const int64_t r1 = min(N, r0 + rows_per_chunk);
  double acc[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[u][v] = 0.0;
  if (l0 < ma && c0 < nb) {
    for (int64_t i = r0; i < r1; ++i) {
      double a[4], bv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] = (l0 + u < ma) ? double(A[i * lda + l0 + u]) : 0.0;
#pragma unroll
      for (int v = 0; v < 4; ++v) bv[v] = (c0 + v < nb) ? double(B[i * ldb + c0 + v]) : 0.0;
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fma(a[u], bv[v], acc[u][v]);
    }
  }
  double* out = part + chunk * int64_t(ma) * nb;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (l0 + u < ma && c0 + v < nb) out[int64_t(l0 + u) * nb + c0 + v] = acc[u][v];
}

__global__ void reduce_partials_kernel(const double* __restrict__ part, int64_t nparts,
                                       int64_t count, double* __restrict__ out,
                                       float* __restrict__ out32) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= count) return;
  double s = 0.0;
  for (int64_t p = 0; p < nparts; ++p) s += part[p * count + idx];
  if (out != nullptr) out[idx] = s;
  if (out32 != nullptr) out32[idx] = float(s);
}

int64_t gemm_tn_chunks(int64_t N) {
  // enough chunks to fill the GPU with (l tiles x chunks) workgroups
  return std::max<int64_t>(1, std::min<int64_t>(512, (N + 1023) / 1024));
}

void gemm_tn(const float* A, int64_t lda, int ma, const float* B, int64_t ldb, int nb, int64_t N,
             FSpanD part, double* C, float* C32, hipStream_t stream) {
  FD_REQUIRE(ma >= 1 && nb >= 1 && N >= 1, FD_ERR_INVALID_ARG, "internal: gemm_tn shape");
  const int64_t chunks = gemm_tn_chunks(N);
  const int64_t rpc = (N + chunks - 1) / chunks;
  check_span_d(part, size_t(chunks) * ma * nb, "gemm partials");
  dim3 grid(nblk(ma, 64), unsigned(chunks));
  hipLaunchKernelGGL(gemm_tn_partial_kernel, grid, dim3(256), 0, stream, A, lda, ma, B, ldb, nb,
                     N, rpc, part.p);
  FD_LAUNCH_CHECK();
  const int64_t count = int64_t(ma) * nb;
  hipLaunchKernelGGL(reduce_partials_kernel, dim3(nblk(count, 256)), dim3(256), 0, stream, part.p,
                     chunks, count, C, C32);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------ Z = beta Z + alpha Q C
// C: ma x nb float32 row-major (ld nb).  Each workgroup owns 256 / nbp rows,
// thread (row, c) loops over l with C staged in LDS in slices of 128 rows.
__global__ __launch_bounds__(256) void gemm_nn_kernel(const float* __restrict__ Q, int64_t ldq,
                                                      int ma, const float* __restrict__ C, int nb,
                                                      int nbp, float* __restrict__ Z,
                                                      int64_t ldz, int64_t N, float alpha,
                                                      float beta) {
  __shared__ float cs[128 * 64];
  const int rows_per_wg = 256 / nbp;
  const int tr = threadIdx.x / nbp, tc = threadIdx.x % nbp;
  const int64_t i = int64_t(blockIdx.x) * rows_per_wg + tr;
  float acc = 0.f;
  for (int l0 = 0; l0 < ma; l0 += 128) {
    const int len = min(128, ma - l0);
    __syncthreads();
    for (int e = threadIdx.x; e < len * nb; e += 256) cs[e] = C[int64_t(l0) * nb + e];
    __syncthreads();
    if (i < N && tc < nb) {
      const float* q = Q + i * ldq + l0;
      for (int l = 0; l < len; ++l) acc = fmaf(q[l], cs[l * nb + tc], acc);
    }
  }
  if (i < N && tc < nb) {
    float* z = Z + i * ldz + tc;
    *z = (beta == 0.f) ? alpha * acc : fmaf(beta, *z, alpha * acc);
  }
}

void gemm_nn(const float* Q, int64_t ldq, int ma, const float* C, int nb, float* Z, int64_t ldz,
             int64_t N, float alpha, float beta, hipStream_t stream) {
  FD_REQUIRE(ma >= 1 && nb >= 1 && nb <= 64, FD_ERR_INVALID_ARG, "internal: gemm_nn shape");
  int nbp = 1;
  while (nbp < nb) nbp <<= 1;
  const int rows_per_wg = 256 / nbp;
  hipLaunchKernelGGL(gemm_nn_kernel, dim3(nblk(N, rows_per_wg)), dim3(256), 0, stream, Q, ldq, ma,
                     C, nb, nbp, Z, ldz, N, alpha, beta);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------ Cholesky + R^-1
// G (b x b, float64, row-major) = R^T R.  A column whose pivot falls below
// rel_tol times its own norm (numerically inside the span of the earlier
// columns), or whose norm is not positive, is flagged; it gets an identity
// row in R and is excluded from the later eliminations.  Output: Rinv
// (float32, upper triangular, ld b) and flags[b] (1 = replace this column).
__global__ __launch_bounds__(64) void chol_rinv_kernel(const double* __restrict__ G, int b,
                                                       double rel_tol, float* __restrict__ Rinv,
                                                       int* __restrict__ flags) {
  __shared__ double R[64 * 64];
  __shared__ double Ri[64 * 64];
  __shared__ int flag[64];
  const int t = threadIdx.x;
  for (int e = t; e < b * b; e += 64) {
    R[e] = 0.0;
    Ri[e] = 0.0;
  }
  __syncthreads();
  // right-looking Cholesky, one column per step (thread t owns column t)
  for (int k = 0; k < b; ++k) {
    if (t == 0) {
      double diag = G[k * b + k];
      double s = diag;
      for (int l = 0; l < k; ++l) s -= R[l * b + k] * R[l * b + k];
      const bool bad = !(diag > 0.0) || !(s > rel_tol * rel_tol * diag) || !isfinite(s);
      flag[k] = bad ? 1 : 0;
      R[k * b + k] = bad ? 1.0 : sqrt(s);
    }
    __syncthreads();
    if (t > k && t < b) {
      double v = 0.0;
      if (!flag[k]) {
        v = G[k * b + t];
        for (int l = 0; l < k; ++l) v -= R[l * b + k] * R[l * b + t];
        v /= R[k * b + k];
      }
      R[k * b + t] = v;
    }
    __syncthreads();
  }
  // Rinv: solve R X = I column by column (thread t owns column t of X)
  if (t < b) {
    for (int i = t; i >= 0; --i) {
      double v = (i == t) ? 1.0 : 0.0;
      for (int l = i + 1; l <= t; ++l) v -= R[i * b + l] * Ri[l * b + t];
      Ri[i * b + t] = v / R[i * b + i];
    }
  }
  __syncthreads();
  for (int e = t; e < b * b; e += 64) Rinv[e] = float(Ri[e]);
  if (t < b) flags[t] = flag[t];
}

void chol_rinv(const double* G, int b, double rel_tol, float* Rinv, int* flags,
               hipStream_t stream) {
  FD_REQUIRE(b >= 1 && b <= 64, FD_ERR_INVALID_ARG, "internal: chol size");
  hipLaunchKernelGGL(chol_rinv_kernel, dim3(1), dim3(64), 0, stream, G, b, rel_tol, Rinv, flags);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------ random fill
// Counter-based generator: SplitMix64 finalizer (Steele, Lea, Flood 2014) of
// (seed, stream, counter) -> two uniforms -> one normal by Box-Muller.
__device__ __forceinline__ uint64_t splitmix64(uint64_t z) {
  z += 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ float normal_at(uint64_t seed, uint64_t stream, uint64_t counter) {
  const uint64_t h1 = splitmix64(seed ^ splitmix64(stream * 0x632be59bd9b4e019ull + counter));
  const uint64_t h2 = splitmix64(h1);
  const double u1 = (double((h1 >> 11) + 1)) * (1.0 / 9007199254740993.0);  // (0, 1]
  const double u2 = double(h2 >> 11) * (1.0 / 9007199254740992.0);          // [0, 1)
  return float(sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2));
}

// Z[:, c] <- N(0, 1) for every c with flags[c] != 0 (flags == NULL: all columns).
__global__ void fill_normal_kernel(float* __restrict__ Z, int64_t ldz, int64_t N, int nb,
                                   const int* __restrict__ flags, uint64_t seed,
                                   uint64_t stream_id) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= N * nb) return;
  const int64_t i = idx / nb;
  const int c = int(idx % nb);
  if (flags != nullptr && flags[c] == 0) return;
  Z[i * ldz + c] = normal_at(seed, stream_id * 64 + uint64_t(c), uint64_t(i));
}

void fill_normal(float* Z, int64_t ldz, int64_t N, int nb, const int* flags, uint64_t seed,
                 uint64_t stream_id, hipStream_t stream) {
  hipLaunchKernelGGL(fill_normal_kernel, dim3(nblk(N * nb, 256)), dim3(256), 0, stream, Z, ldz, N,
                     nb, flags, seed, stream_id);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------ residual norms
// r_c^2 = sum_i (W[i, c] - theta_c Y[i, c])^2 for c < nc, float64 partials.
__global__ __launch_bounds__(256) void residual_partial_kernel(
    const float* __restrict__ Y, const float* __restrict__ W, int64_t ld, int nc,
    const double* __restrict__ theta, int64_t N, int64_t rows_per_chunk,
    double* __restrict__ part) {
  __shared__ double red[256];
  const int c = blockIdx.x;
  const int64_t r0 = int64_t(blockIdx.y) * rows_per_chunk;
  const int64_t r1 = min(N, r0 + rows_per_chunk);
  const double th = theta[c];
  double s = 0.0;
  for (int64_t i = r0 + threadIdx.x; i < r1; i += 256) {
    const double e = double(W[i * ld + c]) - th * double(Y[i * ld + c]);
    s += e * e;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (int(threadIdx.x) < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[int64_t(blockIdx.y) * nc + c] = red[0];
}

__global__ void sqrt_sum_kernel(const double* __restrict__ part, int64_t nparts, int nc,
                                double* __restrict__ out) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nc) return;
  double s = 0.0;
  for (int64_t p = 0; p < nparts; ++p) s += part[p * nc + c];
  out[c] = sqrt(s);
}

void residual_norms(const float* Y, const float* W, int64_t ld, int nc, const double* theta,
                    int64_t N, FSpanD part, double* out, hipStream_t stream) {
  const int64_t chunks = std::max<int64_t>(1, std::min<int64_t>(64, (N + 4095) / 4096));
  const int64_t rpc = (N + chunks - 1) / chunks;
  check_span_d(part, size_t(chunks) * nc, "residual partials");
  hipLaunchKernelGGL(residual_partial_kernel, dim3(unsigned(nc), unsigned(chunks)), dim3(256), 0,
                     stream, Y, W, ld, nc, theta, N, rpc, part.p);
  FD_LAUNCH_CHECK();
  hipLaunchKernelGGL(sqrt_sum_kernel, dim3(nblk(nc, 64)), dim3(64), 0, stream, part.p, chunks, nc,
                     out);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------ Jacobi eigensolver
// Cyclic two-sided Jacobi (Golub & Van Loan, Alg. 8.5.3, parallel ordering):
// in each round the indices are split into disjoint pairs by the circle
// method, every pair (p, q) gets the rotation that annihilates A_pq
// (Alg. 8.5.2), all row rotations are applied, then all column rotations and
// the eigenvector updates.  A (m x m, float64, ld lda) is overwritten; on exit
// theta (m) holds the eigenvalues sorted descending and S (m x m, ld lds) the
// matching eigenvectors in its columns.  Vw (m x m) is a scratch matrix.
__global__ __launch_bounds__(1024) void jacobi_kernel(double* __restrict__ A, int m, int lda,
                                                      double* __restrict__ Vw,
                                                      double* __restrict__ theta,
                                                      double* __restrict__ S, int lds,
                                                      int max_sweeps, double tol,
                                                      int* __restrict__ sweeps_out) {
  __shared__ int pp[512], qq[512];
  __shared__ double cc[512], ss[512];
  __shared__ double red[1024];
  __shared__ int stop;
  const int t = threadIdx.x;
  const int nt = blockDim.x;
  const int me = m + (m & 1);  // even number of players (index m is a dummy when m is odd)
  const int npairs = me / 2;
  for (int e = t; e < m * m; e += nt) Vw[(e / m) * m + (e % m)] = (e / m == e % m) ? 1.0 : 0.0;
  if (t == 0) stop = 0;
  __syncthreads();
  int sweep = 0;
  for (; sweep < max_sweeps; ++sweep) {
    // convergence: off-diagonal Frobenius norm relative to the whole matrix
    double off = 0.0, all = 0.0;
    for (int e = t; e < m * m; e += nt) {
      const int i = e / m, j = e % m;
      const double v = A[int64_t(i) * lda + j];
      all += v * v;
      if (i != j) off += v * v;
    }
    red[t] = off;
    __syncthreads();
    for (int w = nt / 2; w > 0; w >>= 1) {
      if (t < w) red[t] += red[t + w];
      __syncthreads();
    }
    const double off_sum = red[0];
    __syncthreads();
    red[t] = all;
    __syncthreads();
    for (int w = nt / 2; w > 0; w >>= 1) {
      if (t < w) red[t] += red[t + w];
      __syncthreads();
    }
    if (t == 0) stop = (off_sum <= tol * tol * red[0]) ? 1 : 0;
    __syncthreads();
    if (stop) break;
    for (int round = 0; round < me - 1; ++round) {
      for (int k = t; k < npairs; k += nt) {
        // circle method: player 0 fixed, players 1..me-1 rotate
        const int a = (k == 0) ? 0 : ((round + k - 1) % (me - 1)) + 1;
        const int bq = ((round + me - 2 - k) % (me - 1)) + 1;
        int p = min(a, bq), q = max(a, bq);
        double c = 1.0, s = 0.0;
        if (q < m) {
          const double apq = A[int64_t(p) * lda + q];
          if (apq != 0.0) {
            const double app = A[int64_t(p) * lda + p], aqq = A[int64_t(q) * lda + q];
            const double tau = (aqq - app) / (2.0 * apq);
            const double tt = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
            c = 1.0 / sqrt(1.0 + tt * tt);
            s = tt * c;
          }
        } else {
          p = q = -1;
        }
        pp[k] = p;
        qq[k] = q;
        cc[k] = c;
        ss[k] = s;
      }
      __syncthreads();
      // rows: A_p <- c A_p - s A_q, A_q <- s A_p + c A_q
      for (int e = t; e < npairs * m; e += nt) {
        const int k = e / m, j = e % m;
        const int p = pp[k], q = qq[k];
        if (p < 0 || ss[k] == 0.0) continue;
        const double c = cc[k], s = ss[k];
        const double ap = A[int64_t(p) * lda + j], aq = A[int64_t(q) * lda + j];
        A[int64_t(p) * lda + j] = c * ap - s * aq;
        A[int64_t(q) * lda + j] = s * ap + c * aq;
      }
      __syncthreads();
      // columns of A and of V
      for (int e = t; e < npairs * m; e += nt) {
        const int k = e / m, i = e % m;
        const int p = pp[k], q = qq[k];
        if (p < 0 || ss[k] == 0.0) continue;
        const double c = cc[k], s = ss[k];
        const double ap = A[int64_t(i) * lda + p], aq = A[int64_t(i) * lda + q];
        A[int64_t(i) * lda + p] = c * ap - s * aq;
        A[int64_t(i) * lda + q] = s * ap + c * aq;
        const double vp = Vw[int64_t(i) * m + p], vq = Vw[int64_t(i) * m + q];
        Vw[int64_t(i) * m + p] = c * vp - s * vq;
        Vw[int64_t(i) * m + q] = s * vp + c * vq;
      }
      __syncthreads();
    }
  }
  // sort descending: rank of i = number of j before it in the order
  for (int i = t; i < m; i += nt) {
    const double di = A[int64_t(i) * lda + i];
    int rank = 0;
    for (int j = 0; j < m; ++j) {
      const double dj = A[int64_t(j) * lda + j];
      rank += (dj > di || (dj == di && j < i)) ? 1 : 0;
    }
    theta[rank] = di;
    for (int r = 0; r < m; ++r) S[int64_t(r) * lds + rank] = Vw[int64_t(r) * m + i];
  }
  if (t == 0 && sweeps_out != nullptr) *sweeps_out = sweep;
}

void jacobi_eig(double* A, int m, int lda, double* Vw, double* theta, double* S, int lds,
                int* sweeps, hipStream_t stream) {
  FD_REQUIRE(m >= 1 && m <= 1024, FD_ERR_UNSUPPORTED, "projected matrix larger than 1024");
  hipLaunchKernelGGL(jacobi_kernel, dim3(1), dim3(1024), 0, stream, A, m, lda, Vw, theta, S, lds,
                     60, 1e-13, sweeps);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------ small helpers

// dst[i * ldd + c] = src[i * lds + c] * (scale ? scale[i]^power : 1), c < nc
__global__ void copy_cols_kernel(const float* __restrict__ src, int64_t lds, float* __restrict__ dst,
                                 int64_t ldd, int64_t N, int nc, const float* __restrict__ scale,
                                 double power) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= N * nc) return;
  const int64_t i = idx / nc;
  const int c = int(idx % nc);
  float v = src[i * lds + c];
  if (scale != nullptr) v = float(double(v) * pow(double(scale[i]), power));
  dst[i * ldd + c] = v;
}

void copy_cols(const float* src, int64_t lds, float* dst, int64_t ldd, int64_t N, int nc,
               const float* scale, double power, hipStream_t stream) {
  if (N * nc == 0) return;
  hipLaunchKernelGGL(copy_cols_kernel, dim3(nblk(N * nc, 256)), dim3(256), 0, stream, src, lds,
                     dst, ldd, N, nc, scale, power);
  FD_LAUNCH_CHECK();
}

// W[:, c] -= theta_c Y[:, c] in place (turns Ritz images into residuals)
__global__ void sub_theta_kernel(const float* __restrict__ Y, float* __restrict__ W, int64_t ld,
                                 int64_t N, int nc, const double* __restrict__ theta) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= N * nc) return;
  const int64_t i = idx / nc;
  const int c = int(idx % nc);
  W[i * ld + c] = float(double(W[i * ld + c]) - theta[c] * double(Y[i * ld + c]));
}

void sub_theta(const float* Y, float* W, int64_t ld, int64_t N, int nc, const double* theta,
               hipStream_t stream) {
  hipLaunchKernelGGL(sub_theta_kernel, dim3(nblk(N * nc, 256)), dim3(256), 0, stream, Y, W, ld, N,
                     nc, theta);
  FD_LAUNCH_CHECK();
}

// T[0:m, c0:c0+nb] = C and T[c0:c0+nb, 0:m] = C^T (C: m x nb float64); the
// diagonal block is symmetrised.
__global__ void put_block_kernel(double* __restrict__ T, int ldt, const double* __restrict__ C,
                                 int m, int c0, int nb) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= m * nb) return;
  const int r = idx / nb, c = idx % nb;
  double v = C[idx];
  if (r >= c0 && r < c0 + nb) {  // diagonal block: average with the transpose
    const double w = C[int64_t(c0 + c) * nb + (r - c0)];
    v = 0.5 * (v + w);
  }
  T[int64_t(r) * ldt + c0 + c] = v;
  T[int64_t(c0 + c) * ldt + r] = v;
}

void put_block(double* T, int ldt, const double* C, int m, int c0, int nb, hipStream_t stream) {
  hipLaunchKernelGGL(put_block_kernel, dim3(nblk(int64_t(m) * nb, 256)), dim3(256), 0, stream, T,
                     ldt, C, m, c0, nb);
  FD_LAUNCH_CHECK();
}

// T = diag(theta[0:kk]) in the leading m_max x m_max block (rest zero)
__global__ void set_diag_kernel(double* __restrict__ T, int ldt, int mm,
                                const double* __restrict__ theta, int kk) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= mm * mm) return;
  const int r = idx / mm, c = idx % mm;
  T[int64_t(r) * ldt + c] = (r == c && r < kk) ? theta[r] : 0.0;
}

void set_diag(double* T, int ldt, int mm, const double* theta, int kk, hipStream_t stream) {
  hipLaunchKernelGGL(set_diag_kernel, dim3(nblk(int64_t(mm) * mm, 256)), dim3(256), 0, stream, T,
                     ldt, mm, theta, kk);
  FD_LAUNCH_CHECK();
}

// S32[r][c] = float(S[r][c]) for r < m, c < nc  (ld of S32 = nc)
__global__ void narrow_kernel(const double* __restrict__ S, int lds, int m, int nc,
                              float* __restrict__ S32) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= m * nc) return;
  const int r = idx / nc, c = idx % nc;
  S32[idx] = float(S[int64_t(r) * lds + c]);
}

void narrow(const double* S, int lds, int m, int nc, float* S32, hipStream_t stream) {
  hipLaunchKernelGGL(narrow_kernel, dim3(nblk(int64_t(m) * nc, 256)), dim3(256), 0, stream, S, lds,
                     m, nc, S32);
  FD_LAUNCH_CHECK();
}

// copy the matrix block src[0:m, 0:m] (ld lds) to dst (ld ldd)
__global__ void copy_square_kernel(const double* __restrict__ src, int lds, double* __restrict__ dst,
                                   int ldd, int m) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= m * m) return;
  const int r = idx / m, c = idx % m;
  dst[int64_t(r) * ldd + c] = src[int64_t(r) * lds + c];
}

void copy_square(const double* src, int lds, double* dst, int ldd, int m, hipStream_t stream) {
  hipLaunchKernelGGL(copy_square_kernel, dim3(nblk(int64_t(m) * m, 256)), dim3(256), 0, stream, src,
                     lds, dst, ldd, m);
  FD_LAUNCH_CHECK();
}

}  // namespace fd

namespace fd {

// Z[:, j] = W[:, sel[j]] - theta[sel[j]] Q[:, sel[j]] for j < nsel (residual
// vectors of chosen Ritz pairs); Q and W share ld.
__global__ void gather_residuals_kernel(const float* __restrict__ Q, const float* __restrict__ W,
                                        int64_t ld, const double* __restrict__ theta,
                                        const int* __restrict__ sel, int nsel,
                                        float* __restrict__ Z, int64_t ldz, int64_t N) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= N * nsel) return;
  const int64_t i = idx / nsel;
  const int j = int(idx % nsel);
  const int c = sel[j];
  Z[i * ldz + j] = float(double(W[i * ld + c]) - theta[c] * double(Q[i * ld + c]));
}

void gather_residuals(const float* Q, const float* W, int64_t ld, const double* theta,
                      const int* sel, int nsel, float* Z, int64_t ldz, int64_t N,
                      hipStream_t stream) {
  if (nsel <= 0) return;
  hipLaunchKernelGGL(gather_residuals_kernel, dim3(nblk(N * nsel, 256)), dim3(256), 0, stream, Q, W,
                     ld, theta, sel, nsel, Z, ldz, N);
  FD_LAUNCH_CHECK();
}

// Q[i, c] = (i == c) for i < N, c < nc
__global__ void set_identity_kernel(float* __restrict__ Q, int64_t ld, int64_t N, int nc) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= N * nc) return;
  const int64_t i = idx / nc;
  const int c = int(idx % nc);
  Q[i * ld + c] = (i == c) ? 1.f : 0.f;
}

void set_identity(float* Q, int64_t ld, int64_t N, int nc, hipStream_t stream) {
  hipLaunchKernelGGL(set_identity_kernel, dim3(nblk(N * nc, 256)), dim3(256), 0, stream, Q, ld, N,
                     nc);
  FD_LAUNCH_CHECK();
}

}  // namespace fd
