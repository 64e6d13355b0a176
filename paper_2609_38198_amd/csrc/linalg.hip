// Dense helpers of the block Lanczos eigensolver, all on the device:
//   * tall-skinny products C = A^T B (reduction over N rows, float64 partial
//     sums reduced in a fixed order) and Z = beta Z + alpha Q C,
//   * Cholesky of a small Gram matrix with detection of dependent columns,
//   * refill of such columns from a counter-based normal generator,
//   * residual norms ||W s - theta Q s|| of Ritz pairs,
//   * cyclic Jacobi eigensolver for the small symmetric projected matrix.
// Everything is deterministic: no atomics, fixed reduction orders.
#include <algorithm>
#include <cmath>

#include "fd_linalg.hpp"

namespace fd {

static inline unsigned nblk(int64_t n, int t) { return unsigned((n + t - 1) / t); }

// ------------------------------------------------------------ C = A^T B
// Grid (l tiles of 64, row chunks).  Thread (lg, cg) accumulates a 4 x 4
// block C[l0 + 4 lg + u][4 cg + v] in float64 over its chunk of rows, four
// rows per step with all sixteen loads of a step issued before its FMAs.
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
    // columns past the edge read a valid column; their sums are not stored
    int la[4], cb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      la[u] = min(l0 + u, ma - 1);
      cb[u] = min(c0 + u, nb - 1);
    }
    int64_t i = r0;
    for (; i + 4 <= r1; i += 4) {
      float a[4][4], bv[4][4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          a[r][u] = A[(i + r) * lda + la[u]];
          bv[r][u] = B[(i + r) * ldb + cb[u]];
        }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            acc[u][v] = fma(double(a[r][u]), double(bv[r][v]), acc[u][v]);
    }
    for (; i < r1; ++i) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          acc[u][v] = fma(double(A[i * lda + la[u]]), double(B[i * ldb + cb[v]]), acc[u][v]);
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
  // enough chunks (of >= 128 rows) to fill the GPU with (l tiles x chunks)
  // workgroups even when there is a single l tile
  return std::max<int64_t>(1, std::min<int64_t>(1024, (N + 127) / 128));
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
// Cyclic two-sided Jacobi (Golub & Van Loan, Alg. 8.5.3, parallel ordering).
// In each round the indices are split into disjoint pairs by the circle
// method and every pair (p, q) gets the rotation that annihilates A_pq
// (Alg. 8.5.2).  Because the pairs of a round are disjoint, the round's
// similarity transform acts on A block by block: for row pair i and column
// pair j the 2 x 2 block (rows p_i, q_i; columns p_j, q_j) becomes
// R_i^T X R_j.  One launch per round does all blocks (and the matching
// column rotations of the eigenvector matrix) with as many workgroups as the
// size needs, reading A and writing its transform to a second buffer; every
// workgroup recomputes the round's rotations from the (unchanged) input.
// After each sweep the off-diagonal Frobenius norm is checked on the host
// (one scalar read back).  On exit theta (m) holds the eigenvalues sorted
// descending and S (m x m, ld lds) the matching eigenvectors in its columns.

// pair k of round `round` among me (even) players: indices p < q, q = -1 for
// the dummy player of an odd m; rotation (c, s) annihilating A_pq
__device__ __forceinline__ void jacobi_pair(const double* __restrict__ A, int lda, int m, int me,
                                            int round, int k, int& p, int& q, double& c,
                                            double& s) {
  const int a = (k == 0) ? 0 : ((round + k - 1) % (me - 1)) + 1;
  const int bq = ((round + me - 2 - k) % (me - 1)) + 1;
  p = min(a, bq);
  q = max(a, bq);
  c = 1.0;
  s = 0.0;
  if (q >= m) {
    q = -1;  // dummy partner: identity
    return;
  }
  const double apq = A[int64_t(p) * lda + q];
  if (apq != 0.0) {
    const double app = A[int64_t(p) * lda + p], aqq = A[int64_t(q) * lda + q];
    const double tau = (aqq - app) / (2.0 * apq);
    const double tt = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
    c = 1.0 / sqrt(1.0 + tt * tt);
    s = tt * c;
  }
}

// One round: B = J^T A J block by block, V <- V J (in place).
__global__ __launch_bounds__(256) void jacobi_round_kernel(const double* __restrict__ A,
                                                           double* __restrict__ B, int lda,
                                                           double* __restrict__ V, int m, int me,
                                                           int round) {
  __shared__ int pp[512], qq[512];
  __shared__ double cc[512], ss[512];
  const int npairs = me / 2;
  for (int k = threadIdx.x; k < npairs; k += blockDim.x) {
    int p, q;
    double c, s;
    jacobi_pair(A, lda, m, me, round, k, p, q, c, s);
    pp[k] = p;
    qq[k] = q;
    cc[k] = c;
    ss[k] = s;
  }
  __syncthreads();
  const int64_t nA = int64_t(npairs) * npairs;
  const int64_t nV = int64_t(m) * npairs;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < nA + nV; idx += stride) {
    if (idx < nA) {
      const int i = int(idx / npairs), j = int(idx % npairs);
      const int pi = pp[i], qi = qq[i], pj = pp[j], qj = qq[j];
      const double ci = cc[i], si = ss[i], cj = cc[j], sj = ss[j];
      const double a = A[int64_t(pi) * lda + pj];
      const double b = qj >= 0 ? A[int64_t(pi) * lda + qj] : 0.0;
      const double d = qi >= 0 ? A[int64_t(qi) * lda + pj] : 0.0;
      const double e = (qi >= 0 && qj >= 0) ? A[int64_t(qi) * lda + qj] : 0.0;
      // rows: p' = c p - s q, q' = s p + c q; then the same on the columns
      const double a1 = ci * a - si * d, b1 = ci * b - si * e;
      const double d1 = si * a + ci * d, e1 = si * b + ci * e;
      B[int64_t(pi) * lda + pj] = cj * a1 - sj * b1;
      if (qj >= 0) B[int64_t(pi) * lda + qj] = sj * a1 + cj * b1;
      if (qi >= 0) B[int64_t(qi) * lda + pj] = cj * d1 - sj * e1;
      if (qi >= 0 && qj >= 0) B[int64_t(qi) * lda + qj] = sj * d1 + cj * e1;
    } else {
      const int64_t v = idx - nA;
      const int r = int(v / npairs), j = int(v % npairs);
      const int pj = pp[j], qj = qq[j];
      if (qj < 0 || ss[j] == 0.0) continue;
      const double cj = cc[j], sj = ss[j];
      const double vp = V[int64_t(r) * m + pj], vq = V[int64_t(r) * m + qj];
      V[int64_t(r) * m + pj] = cj * vp - sj * vq;
      V[int64_t(r) * m + qj] = sj * vp + cj * vq;
    }
  }
}

__global__ void jacobi_init_kernel(double* __restrict__ V, int m) {
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e < int64_t(m) * m) V[e] = (e / m == e % m) ? 1.0 : 0.0;
}

// out[0] = sum of squared off-diagonal entries, out[1] = sum of all (one
// workgroup, fixed order)
__global__ __launch_bounds__(1024) void jacobi_offnorm_kernel(const double* __restrict__ A, int m,
                                                              int lda, double* __restrict__ out) {
  __shared__ double r0[1024], r1[1024];
  const int t = threadIdx.x;
  double off = 0.0, all = 0.0;
  for (int64_t e = t; e < int64_t(m) * m; e += blockDim.x) {
    const int i = int(e / m), j = int(e % m);
    const double v = A[int64_t(i) * lda + j];
    all += v * v;
    if (i != j) off += v * v;
  }
  r0[t] = off;
  r1[t] = all;
  __syncthreads();
  for (int w = blockDim.x / 2; w > 0; w >>= 1) {
    if (t < w) {
      r0[t] += r0[t + w];
      r1[t] += r1[t + w];
    }
    __syncthreads();
  }
  if (t == 0) {
    out[0] = r0[0];
    out[1] = r1[0];
  }
}

// theta = diag(A) sorted descending, S columns = matching columns of V
__global__ void jacobi_sort_kernel(const double* __restrict__ A, int m, int lda,
                                   const double* __restrict__ V, double* __restrict__ theta,
                                   double* __restrict__ S, int lds) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  const double di = A[int64_t(i) * lda + i];
  int rank = 0;
  for (int j = 0; j < m; ++j) {
    const double dj = A[int64_t(j) * lda + j];
    rank += (dj > di || (dj == di && j < i)) ? 1 : 0;
  }
  theta[rank] = di;
  for (int r = 0; r < m; ++r) S[int64_t(r) * lds + rank] = V[int64_t(r) * m + i];
}

void jacobi_eig(double* A, double* A2, int m, int lda, double* Vw, double* theta, double* S,
                int lds, double* norms, hipStream_t stream) {
  FD_REQUIRE(m >= 1 && m <= 1024, FD_ERR_UNSUPPORTED, "projected matrix larger than 1024");
  constexpr int MAX_SWEEPS = 60;
  constexpr double TOL = 1e-13;
  const int me = m + (m & 1);
  const int npairs = me / 2;
  const int64_t items = int64_t(npairs) * npairs + int64_t(m) * npairs;
  const unsigned grid = unsigned(std::min<int64_t>(2048, std::max<int64_t>(1, (items + 255) / 256)));
  hipLaunchKernelGGL(jacobi_init_kernel, dim3(nblk(int64_t(m) * m, 256)), dim3(256), 0, stream, Vw,
                     m);
  FD_LAUNCH_CHECK();
  double* cur = A;
  double* nxt = A2;
  for (int sweep = 0; sweep < MAX_SWEEPS && m > 1; ++sweep) {
    hipLaunchKernelGGL(jacobi_offnorm_kernel, dim3(1), dim3(1024), 0, stream, cur, m, lda, norms);
    FD_LAUNCH_CHECK();
    double h[2] = {0.0, 0.0};
    FD_HIP_CHECK(hipMemcpyAsync(h, norms, sizeof(h), hipMemcpyDeviceToHost, stream));
    FD_HIP_CHECK(hipStreamSynchronize(stream));
    if (h[0] <= TOL * TOL * h[1]) break;
    for (int round = 0; round < me - 1; ++round) {
      hipLaunchKernelGGL(jacobi_round_kernel, dim3(grid), dim3(256), 0, stream, cur, nxt, lda, Vw,
                         m, me, round);
      FD_LAUNCH_CHECK();
      std::swap(cur, nxt);
    }
  }
  hipLaunchKernelGGL(jacobi_sort_kernel, dim3(nblk(m, 256)), dim3(256), 0, stream, cur, m, lda, Vw,
                     theta, S, lds);
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
