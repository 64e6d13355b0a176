// Dense helpers of the block Lanczos eigensolver, all on the device:
//   * tall-skinny products C = A^T B (reduction over N rows, float64 partial
//     sums reduced in a fixed order) and Z = beta Z + alpha Q C,
//   * Cholesky of a small Gram matrix with detection of dependent columns,
//   * refill of such columns from a counter-based normal generator,
//   * residual norms ||W s - theta Q s|| of Ritz pairs,
//   * parallel cyclic Jacobi eigensolver for the small symmetric projected
//     matrix.
// Everything is deterministic: no atomics, fixed reduction orders.
#include <algorithm>
#include <cmath>

#include "fd_linalg.hpp"

namespace fd {

static inline unsigned nblk(int64_t n, int t) { return unsigned((n + t - 1) / t); }

// ------------------------------------------------------------ C = A^T B
// Each thread accumulates a 4 x 4 block C[4 lq + u][4 cq + v] in float64
// (products of float32 values are exact in float64).  The output is split
// into groups of lqg x tc such blocks (tc = ceil(nb / 4) column quads, lqg
// row quads, at most 256 threads); a workgroup of 256 threads holds
// S = 256 / (lqg tc) slices of one group, which walk interleaved 4-row steps
// of the workgroup's chunk of rows and are added in LDS in slice order.  Grid
// (groups, chunks); partial sums per chunk are then reduced in a fixed order.

struct GemmTnShape {
  int tc = 1, lqg = 1, slices = 1, groups = 1;
  int64_t chunks = 1, rows_per_chunk = 1;
};

static GemmTnShape gemm_tn_shape(int ma, int nb, int64_t N) {
  GemmTnShape g;
  g.tc = (nb + 3) / 4;
  const int lq = (ma + 3) / 4;
  g.lqg = std::min(lq, 256 / g.tc);
  g.groups = (lq + g.lqg - 1) / g.lqg;
  g.lqg = (lq + g.groups - 1) / g.groups;  // balance the groups
  g.slices = 256 / (g.lqg * g.tc);
  // 4 to 16 steps of 4 rows per thread (a multiple of the 4 a loop iteration
  // takes): as few as keep >= ~512 workgroups busy, but at most
  // gemm_tn_chunks(N) chunks (the partial buffer's size)
  const int64_t steps_total = (N + 3) / 4;
  int64_t spt = steps_total * g.groups / (int64_t(g.slices) * 512);
  spt = round_up(std::max<int64_t>(4, std::min<int64_t>(16, spt)), 4);
  g.rows_per_chunk = 4 * spt * g.slices;
  g.chunks = (N + g.rows_per_chunk - 1) / g.rows_per_chunk;
  const int64_t cap = gemm_tn_chunks(N);
  if (g.chunks > cap) {
    g.chunks = cap;
    g.rows_per_chunk = round_up((N + cap - 1) / cap, int64_t(4) * g.slices);
    g.chunks = (N + g.rows_per_chunk - 1) / g.rows_per_chunk;
  }
  return g;
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

// VEC: ma, nb, lda, ldb multiples of 4 and A, B 16-byte aligned; each step
// then reads its 4 + 4 values per row as two 16-byte loads (same sums).
template <bool VEC>
__global__ __launch_bounds__(256) void gemm_tn_partial_kernel(
    const float* __restrict__ A, int64_t lda, int ma, const float* __restrict__ B, int64_t ldb,
    int nb, int64_t N, int64_t rows_per_chunk, int tc, int lqg, int slices,
    double* __restrict__ part) {
  __shared__ double red[256 * 16];
  const int t = threadIdx.x;
  const int to = lqg * tc;
  const int slice = t / to, o = t % to;
  const int l0 = 4 * (blockIdx.x * lqg + o / tc);
  const int c0 = 4 * (o % tc);
  const bool active = slice < slices && l0 < ma;
  const int64_t chunk = blockIdx.y;
  const int64_t r0 = chunk * rows_per_chunk;
  const int64_t r1 = min(N, r0 + rows_per_chunk);
  double acc[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[u][v] = 0.0;
  if (active) {
    // columns past the edge read a valid column; their sums are not stored
    int la[4], cb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      la[u] = min(l0 + u, ma - 1);
      cb[u] = min(c0 + u, nb - 1);
    }
    // four steps (of 4 rows) per iteration with all their loads issued first:
    // the rows are far apart in memory and each step alone would wait a full
    // load latency; rows past the chunk read its last row with weight 0
    const int64_t stride = 4 * int64_t(slices);
    for (int64_t i = r0 + 4 * slice; i < r1; i += 4 * stride) {
      float a[4][4][4], bv[4][4][4];
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t ir = i + st * stride + r;
          const int64_t irc = min(ir, r1 - 1);
          if constexpr (VEC) {
            const f32x4 av = *reinterpret_cast<const f32x4*>(A + irc * lda + l0);
            const f32x4 bw = *reinterpret_cast<const f32x4*>(B + irc * ldb + c0);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              a[st][r][u] = av[u];
              bv[st][r][u] = (ir < r1) ? bw[u] : 0.f;
            }
          } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              a[st][r][u] = A[irc * lda + la[u]];
              bv[st][r][u] = (ir < r1) ? B[irc * ldb + cb[u]] : 0.f;
            }
          }
        }
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int v = 0; v < 4; ++v)
              acc[u][v] = fma(double(a[st][r][u]), double(bv[st][r][v]), acc[u][v]);
    }
  }
  if (slices > 1) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[(4 * u + v) * 256 + t] = acc[u][v];
    __syncthreads();
    if (slice == 0) {
      for (int sl = 1; sl < slices; ++sl)
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v) acc[u][v] += red[(4 * u + v) * 256 + sl * to + o];
    }
  }
  if (slice != 0 || !active) return;
  double* out = part + chunk * int64_t(ma) * nb;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (l0 + u < ma && c0 + v < nb) out[int64_t(l0 + u) * nb + c0 + v] = acc[u][v];
}

// out[idx] = sum over p of part[p * count + idx]: 8 threads per output, each
// summing every 8th partial, then added in thread order (fixed).
__global__ __launch_bounds__(256) void reduce_partials_kernel(const double* __restrict__ part,
                                                              int64_t nparts, int64_t count,
                                                              double* __restrict__ out,
                                                              float* __restrict__ out32) {
  __shared__ double red[8][32];
  const int lane = threadIdx.x & 31, team = threadIdx.x >> 5;
  const int64_t idx = int64_t(blockIdx.x) * 32 + lane;
  double s = 0.0;
  if (idx < count)
    for (int64_t p = team; p < nparts; p += 8) s += part[p * count + idx];
  red[team][lane] = s;
  __syncthreads();
  if (team != 0 || idx >= count) return;
  double tot = red[0][lane];
  for (int k = 1; k < 8; ++k) tot += red[k][lane];
  if (out != nullptr) out[idx] = tot;
  if (out32 != nullptr) out32[idx] = float(tot);
}

int64_t gemm_tn_chunks(int64_t N) {
  // bound on the row chunks of gemm_tn (its partial buffer holds this many)
  return std::max<int64_t>(1, std::min<int64_t>(1024, (N + 15) / 16));
}

void gemm_tn(const float* A, int64_t lda, int ma, const float* B, int64_t ldb, int nb, int64_t N,
             FSpanD part, double* C, float* C32, hipStream_t stream) {
  FD_REQUIRE(ma >= 1 && nb >= 1 && nb <= 64 && N >= 1, FD_ERR_INVALID_ARG,
             "internal: gemm_tn shape");
  const GemmTnShape g = gemm_tn_shape(ma, nb, N);
  check_span_d(part, size_t(g.chunks) * ma * nb, "gemm partials");
  const bool vec = ma % 4 == 0 && nb % 4 == 0 && lda % 4 == 0 && ldb % 4 == 0 &&
                   reinterpret_cast<uintptr_t>(A) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(B) % 16 == 0;
  const dim3 grid(unsigned(g.groups), unsigned(g.chunks));
  if (vec)
    hipLaunchKernelGGL(gemm_tn_partial_kernel<true>, grid, dim3(256), 0, stream, A, lda, ma, B, ldb,
                       nb, N, g.rows_per_chunk, g.tc, g.lqg, g.slices, part.p);
  else
    hipLaunchKernelGGL(gemm_tn_partial_kernel<false>, grid, dim3(256), 0, stream, A, lda, ma, B,
                       ldb, nb, N, g.rows_per_chunk, g.tc, g.lqg, g.slices, part.p);
  FD_LAUNCH_CHECK();
  const int64_t count = int64_t(ma) * nb;
  hipLaunchKernelGGL(reduce_partials_kernel, dim3(nblk(count, 32)), dim3(256), 0, stream, part.p,
                     g.chunks, count, C, C32);
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

// Same product with ma, nb, ldq, ldz multiples of 4 and Q, Z 16-byte aligned:
// thread (row, column quad) reads its row of Q four values at a time and
// writes four outputs at once; every output is the same fmaf chain over l in
// order as in gemm_nn_kernel.
__global__ __launch_bounds__(256) void gemm_nn4_kernel(const float* __restrict__ Q, int64_t ldq,
                                                       int ma, const float* __restrict__ C, int nb,
                                                       int nqp, float* __restrict__ Z, int64_t ldz,
                                                       int64_t N, float alpha, float beta) {
  __shared__ float cs[128 * 64];
  const int rows_per_wg = 256 / nqp;
  const int tr = threadIdx.x / nqp, tq = threadIdx.x % nqp;
  const int64_t i = int64_t(blockIdx.x) * rows_per_wg + tr;
  const bool active = i < N && 4 * tq < nb;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int l0 = 0; l0 < ma; l0 += 128) {
    const int len = min(128, ma - l0);
    __syncthreads();
    for (int e = threadIdx.x; e < len * nb; e += 256) cs[e] = C[int64_t(l0) * nb + e];
    __syncthreads();
    if (active) {
      const float* q = Q + i * ldq + l0;
      for (int l = 0; l < len; l += 4) {
        const f32x4 q4 = *reinterpret_cast<const f32x4*>(q + l);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const f32x4 c4 = *reinterpret_cast<const f32x4*>(cs + (l + u) * nb + 4 * tq);
#pragma unroll
          for (int v = 0; v < 4; ++v) acc[v] = fmaf(q4[u], c4[v], acc[v]);
        }
      }
    }
  }
  if (active) {
    f32x4* z = reinterpret_cast<f32x4*>(Z + i * ldz + 4 * tq);
    f32x4 out;
    if (beta == 0.f) {
#pragma unroll
      for (int v = 0; v < 4; ++v) out[v] = alpha * acc[v];
    } else {
      const f32x4 zo = *z;
#pragma unroll
      for (int v = 0; v < 4; ++v) out[v] = fmaf(beta, zo[v], alpha * acc[v]);
    }
    *z = out;
  }
}

void gemm_nn(const float* Q, int64_t ldq, int ma, const float* C, int nb, float* Z, int64_t ldz,
             int64_t N, float alpha, float beta, hipStream_t stream) {
  FD_REQUIRE(ma >= 1 && nb >= 1 && nb <= 64, FD_ERR_INVALID_ARG, "internal: gemm_nn shape");
  if (ma % 4 == 0 && nb % 4 == 0 && ldq % 4 == 0 && ldz % 4 == 0 &&
      reinterpret_cast<uintptr_t>(Q) % 16 == 0 && reinterpret_cast<uintptr_t>(Z) % 16 == 0) {
    int nqp = 1;
    while (nqp < nb / 4) nqp <<= 1;
    hipLaunchKernelGGL(gemm_nn4_kernel, dim3(nblk(N, 256 / nqp)), dim3(256), 0, stream, Q, ldq,
                       ma, C, nb, nqp, Z, ldz, N, alpha, beta);
    FD_LAUNCH_CHECK();
    return;
  }
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
// R_i^T X R_j.  Two ways to run the rounds:
//   * m <= JL_MAX: one workgroup holds the upper triangle in LDS and runs
//     whole sweeps with a barrier between rounds (jacobi_lds_kernel); the
//     rotations are logged and replayed on the eigenvector matrix by a
//     second kernel (jacobi_replay_kernel);
//   * larger m: one launch per round does all blocks (and the matching
//     column rotations of the eigenvector matrix) with as many workgroups as
//     the size needs, reading A and writing its transform to a second buffer;
//     every workgroup recomputes the round's rotations from the (unchanged)
//     input, and after each sweep the off-diagonal Frobenius norm is checked
//     on the host (one scalar read back).
// On exit theta (m) holds the eigenvalues sorted descending and S (m x m,
// ld lds) the matching eigenvectors in its columns.

// circle-method pair k of round `round` among me players (p < q, q >= m for
// the dummy player of an odd m)
__device__ __forceinline__ void circle_pair(int me, int round, int k, int& p, int& q) {
  const int a = (k == 0) ? 0 : ((round + k - 1) % (me - 1)) + 1;
  const int bq = ((round + me - 2 - k) % (me - 1)) + 1;
  p = min(a, bq);
  q = max(a, bq);
}

// rotation (c, s) annihilating A_pq (apq != 0): t = tan of the angle, the
// smaller root of t^2 + 2 tau t - 1 = 0 (the 2 x 2 symmetric Schur
// decomposition of Golub & Van Loan)
// (with tau = (aqq - app) / (2 apq) multiplied through by 2 |apq|: one square
// root and one division fewer on the dependent chain)
__device__ __forceinline__ void jacobi_rotation(double app, double aqq, double apq, double& c,
                                                double& s) {
  const double d = aqq - app;
  const double tt = (d >= 0.0 ? 2.0 * apq : -2.0 * apq) / (fabs(d) + sqrt(d * d + 4.0 * apq * apq));
  c = rsqrt(1.0 + tt * tt);
  s = tt * c;
}

// pair k of round `round` among me (even) players: indices p < q, q = -1 for
// the dummy player of an odd m; rotation (c, s) annihilating A_pq
__device__ __forceinline__ void jacobi_pair(const double* __restrict__ A, int lda, int m, int me,
                                            int round, int k, int& p, int& q, double& c,
                                            double& s) {
  circle_pair(me, round, k, p, q);
  c = 1.0;
  s = 0.0;
  if (q >= m) {
    q = -1;  // dummy partner: identity
    return;
  }
  const double apq = A[int64_t(p) * lda + q];
  if (apq != 0.0) jacobi_rotation(A[int64_t(p) * lda + p], A[int64_t(q) * lda + q], apq, c, s);
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

// ---- one-workgroup variant for m <= JL_MAX
// The upper triangle of A (float64) fits in one workgroup's LDS, so a single
// workgroup runs whole sweeps with a barrier between rounds instead of a
// launch per round; blocks whose two rotations are both the identity are
// skipped (most of them in the last sweeps).  The rotations (c, s) of every
// round are logged in order; a second kernel replays them on the rows of V
// (rows are independent under column rotations), one workgroup per group of
// rows held in LDS.

constexpr int JL_MAX = 192;   // largest m on the one-workgroup path
constexpr int JL_SWEEPS = 4;  // sweeps per launch (the log holds this many)
constexpr int JL_BATCH = 32;  // rounds of the log staged in LDS at a time by the replay

// log capacity that every size up to m needs
size_t jacobi_log_doubles(int m) {
  const int mc = std::min(m, JL_MAX);
  const int me = mc + (mc & 1);
  return size_t(JL_SWEEPS) * me * std::max(me - 1, 1);
}


// Up to max_sweeps sweeps on A (m x m, ld lda, symmetric; read at the start,
// written back in full at the end).  Stops at the start of a sweep whose
// off-diagonal norm is <= tol * the Frobenius norm.  state[0] = rounds done
// (their rotations in log, me doubles per round: c, s per pair), state[1] = 1
// if converged.  sweep0: sweeps done by earlier launches.  An odd m gets a
// zero row and column m (the circle method's dummy player: its rotations are
// the identity and it stays zero).  From the fifth sweep on, an A_pq
// negligible next to both A_pp and A_qq in float64 (100 |A_pq| vanishes when
// added to either) is set to zero instead of rotated (Rutishauser's rule), so
// late sweeps leave most blocks untouched.
__global__ __launch_bounds__(1024) void jacobi_lds_kernel(double* __restrict__ A, int m, int lda,
                                                          double* __restrict__ log,
                                                          int* __restrict__ state, double tol2,
                                                          int max_sweeps, int sweep0) {
  __shared__ double tri[JL_MAX * (JL_MAX + 1) / 2];
  __shared__ int4 pr[JL_MAX / 2];      // p, q, row offsets of p and q
  __shared__ double2 rot[JL_MAX / 2];  // c, s
  __shared__ double red[2][16];
  const int t = threadIdx.x;
  const int nt = blockDim.x;
  const int me = m + (m & 1), n = me / 2;
  // upper-triangle position of (r, c), r <= c, in the me x me matrix
  auto roff = [me](int r) { return r * me - r * (r + 1) / 2; };
  for (int e = t; e < me * me; e += nt) {
    const int r = e / me, c = e % me;
    if (c >= r) tri[roff(r) + c] = (c < m) ? A[int64_t(r) * lda + c] : 0.0;
  }
  __syncthreads();
  // blocks (i, j), i <= j, folded into groups of n + 1: group g holds the
  // blocks of column pairs g and n - 1 - g (only g for the middle one of an
  // odd n), TPG threads per group
  const int ng = (n + 1) / 2;
  const int tpg = nt / ng;
  const int grp = t / tpg, gl = t % tpg;
  const int gcnt = grp < ng ? (2 * grp + 1 == n ? grp + 1 : n + 1) : 0;
  int rounds = 0, converged = 0;
  for (int sweep = 0; sweep < max_sweeps; ++sweep) {
    // squared off-diagonal and total Frobenius norms (fixed reduction order)
    double off = 0.0, all = 0.0;
    for (int e = t; e < me * me; e += nt) {
      const int r = e / me, c = e % me;
      if (c < r) continue;
      const double v = tri[roff(r) + c];
      if (c == r) {
        all += v * v;
      } else {
        off += 2.0 * v * v;
        all += 2.0 * v * v;
      }
    }
    for (int o = 32; o > 0; o >>= 1) {
      off += __shfl_down(off, o);
      all += __shfl_down(all, o);
    }
    if ((t & 63) == 0) {
      red[0][t >> 6] = off;
      red[1][t >> 6] = all;
    }
    __syncthreads();
    double offs = 0.0, alls = 0.0;
    for (int w = 0; w < nt / 64; ++w) {
      offs += red[0][w];
      alls += red[1][w];
    }
    __syncthreads();  // red is rewritten next sweep
    if (offs <= tol2 * alls) {
      converged = 1;
      break;
    }
    const bool late = sweep0 + sweep >= 4;
    for (int round = 0; round < me - 1; ++round) {
      for (int k = t; k < n; k += nt) {
        int p, q;
        circle_pair(me, round, k, p, q);
        const int rp = roff(p), rq = roff(q);
        const double apq = tri[rp + q], app = tri[rp + p], aqq = tri[rq + q];
        double c = 1.0, s = 0.0;
        const double g = 100.0 * fabs(apq);
        if (late && fabs(app) + g == fabs(app) && fabs(aqq) + g == fabs(aqq)) {
          tri[rp + q] = 0.0;
          } else if (apq != 0.0) {
            jacobi_rotation(app, aqq, apq, c, s);
          }
        pr[k] = make_int4(p, q, rp, rq);
        rot[k] = make_double2(c, s);
        log[(int64_t(rounds) * n + k) * 2] = c;
        log[(int64_t(rounds) * n + k) * 2 + 1] = s;
      }
      __syncthreads();
      // block (i, j): rows p_i, q_i and columns p_j, q_j become R_i^T X R_j;
      // each upper-triangle entry belongs to exactly one block with i <= j
      for (int bk = gl; bk < gcnt; bk += tpg) {
        const int i = bk <= grp ? bk : bk - grp - 1;
        const int j = bk <= grp ? grp : n - 1 - grp;
        // the pair data of both blocks in one go (one LDS wait, not two): the
        // positions are formed before the skip test
        const double2 ri = rot[i], rj = rot[j];
        const int4 Pi = pr[i], Pj = pr[j];
        // position of (r, c) given both row offsets
        auto pos = [](int r, int ro_r, int c, int ro_c) { return r <= c ? ro_r + c : ro_c + r; };
        const int xa = pos(Pi.x, Pi.z, Pj.x, Pj.z), xb = pos(Pi.x, Pi.z, Pj.y, Pj.w);
        const int xd = pos(Pi.y, Pi.w, Pj.x, Pj.z), xe = pos(Pi.y, Pi.w, Pj.y, Pj.w);
        asm volatile("" ::"v"(xa), "v"(xb), "v"(xd), "v"(xe));
        if (ri.y == 0.0 && rj.y == 0.0) continue;
        const double a = tri[xa], b = tri[xb], d = tri[xd], e = tri[xe];
        const double ci = ri.x, si = ri.y, cj = rj.x, sj = rj.y;
        const double a1 = ci * a - si * d, b1 = ci * b - si * e;
        const double d1 = si * a + ci * d, e1 = si * b + ci * e;
        tri[xa] = cj * a1 - sj * b1;
        tri[xb] = sj * a1 + cj * b1;
        if (i != j) tri[xd] = cj * d1 - sj * e1;
        tri[xe] = sj * d1 + cj * e1;
      }
      __syncthreads();
      ++rounds;
    }
  }
  for (int e = t; e < m * m; e += nt) {
    const int r = e / m, c = e % m;
    A[int64_t(r) * lda + c] = r <= c ? tri[roff(r) + c] : tri[roff(c) + r];
  }
  if (t == 0) {
    state[0] = rounds;
    state[1] = converged;
  }
}

// V (m x m, ld m) <- V J_1 J_2 ... for the state[0] logged rounds.  Rows are
// independent under column rotations, so each wave owns one row of V (held
// in LDS) and applies the rounds to it in order with no barrier: lane l takes
// pairs l and l + 64, whose indices it advances from round to round (the
// circle method moves every player but 0 one place per round); within a
// wave LDS accesses complete in order.  The four waves of a workgroup share
// the log, staged in LDS JL_BATCH rounds at a time, the next batch loaded
// into registers while the current one is applied.
__global__ __launch_bounds__(256) void jacobi_replay_kernel(double* __restrict__ V, int m,
                                                            const double* __restrict__ log,
                                                            const int* __restrict__ state) {
  __shared__ double vs[4][JL_MAX];
  __shared__ double stage[2][JL_BATCH * JL_MAX];
  const int t = threadIdx.x;
  const int lane = t & 63, wv = t >> 6;
  const int me = m + (m & 1), n = me / 2;
  const int row = blockIdx.x * 4 + wv;
  const bool active = row < m;
  const int rounds = state[0];
  if (rounds <= 0) return;
  double* v = vs[wv];
  if (active)
    for (int c = lane; c < m; c += 64) v[c] = V[int64_t(row) * m + c];
  // pair indices of round 0 for pairs lane and lane + 64
  int pa[2], pb[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = lane + 64 * h;
    pa[h] = k;            // 0 for k = 0 (player 0 never moves)
    pb[h] = me - 1 - k;
  }
  const int per_batch = JL_BATCH * me;  // doubles of the log per batch
  constexpr int PF = (JL_BATCH * JL_MAX + 255) / 256;  // loads per thread per batch
  const int nbatch = (rounds + JL_BATCH - 1) / JL_BATCH;
  auto fetch = [&](int bt, double (&reg)[PF]) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int e = t + u * 256;
      const int64_t g = int64_t(bt) * per_batch + e;
      reg[u] = (e < per_batch && g < int64_t(rounds) * me) ? log[g] : 0.0;
    }
  };
  auto put = [&](int slot, const double (&reg)[PF]) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int e = t + u * 256;
      if (e < per_batch) stage[slot][e] = reg[u];
    }
  };
  double reg[PF];
  fetch(0, reg);
  put(0, reg);
  __syncthreads();
  for (int bt = 0; bt < nbatch; ++bt) {
    if (bt + 1 < nbatch) fetch(bt + 1, reg);
    const int r1 = min(rounds, (bt + 1) * JL_BATCH);
    const double* sb = stage[bt & 1];
    for (int r = bt * JL_BATCH; r < r1; ++r) {
      // both pairs' reads first (one LDS latency per round), then the writes;
      // the pairs of a round are disjoint, so the two never touch one entry
      int p[2], q[2];
      bool on[2];
      double c[2], sn[2], vp[2], vq[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = lane + 64 * h;
        p[h] = min(pa[h], pb[h]);
        q[h] = max(pa[h], pb[h]);
        on[h] = active && k < n && q[h] < m;
        const int o = ((r - bt * JL_BATCH) * n + min(k, n - 1)) * 2;
        c[h] = sb[o];
        sn[h] = sb[o + 1];
        vp[h] = v[on[h] ? p[h] : 0];
        vq[h] = v[on[h] ? q[h] : 0];
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (on[h] && sn[h] != 0.0) {
          v[p[h]] = c[h] * vp[h] - sn[h] * vq[h];
          v[q[h]] = sn[h] * vp[h] + c[h] * vq[h];
        }
        if (lane + 64 * h != 0) pa[h] = pa[h] == me - 1 ? 1 : pa[h] + 1;
        pb[h] = pb[h] == me - 1 ? 1 : pb[h] + 1;
      }
    }
    if (bt + 1 < nbatch) {
      __syncthreads();  // every wave is done with the slot about to be refilled
      put((bt + 1) & 1, reg);
      __syncthreads();
    }
  }
  if (active)
    for (int c = lane; c < m; c += 64) V[int64_t(row) * m + c] = v[c];
}

void jacobi_eig(double* A, double* A2, int m, int lda, double* Vw, double* theta, double* S,
                int lds, double* norms, FSpanD log, int* state, hipStream_t stream) {
  FD_REQUIRE(m >= 1 && m <= 1024, FD_ERR_UNSUPPORTED, "projected matrix larger than 1024");
  constexpr int MAX_SWEEPS = 60;
  constexpr double TOL = 1e-13;
  const int me = m + (m & 1);
  const int npairs = me / 2;
  hipLaunchKernelGGL(jacobi_init_kernel, dim3(nblk(int64_t(m) * m, 256)), dim3(256), 0, stream, Vw,
                     m);
  FD_LAUNCH_CHECK();
  double* cur = A;
  if (m > 1 && m <= JL_MAX) {
    check_span_d(log, jacobi_log_doubles(m), "jacobi rotation log");
    FD_REQUIRE(lda >= m && state != nullptr, FD_ERR_INVALID_ARG, "internal: jacobi state");
    const unsigned rgrid = unsigned((m + 3) / 4);
    for (int done = 0; done < MAX_SWEEPS; done += JL_SWEEPS) {
      hipLaunchKernelGGL(jacobi_lds_kernel, dim3(1), dim3(1024), 0, stream, A, m, lda, log.p,
                         state, TOL * TOL, std::min(JL_SWEEPS, MAX_SWEEPS - done), done);
      FD_LAUNCH_CHECK();
      hipLaunchKernelGGL(jacobi_replay_kernel, dim3(rgrid), dim3(256), 0, stream, Vw, m, log.p,
                         state);
      FD_LAUNCH_CHECK();
      int h[2] = {0, 0};
      FD_HIP_CHECK(hipMemcpyAsync(h, state, sizeof(h), hipMemcpyDeviceToHost, stream));
      FD_HIP_CHECK(hipStreamSynchronize(stream));
      if (h[1]) break;
    }
  } else {
    const int64_t items = int64_t(npairs) * npairs + int64_t(m) * npairs;
    const unsigned grid =
        unsigned(std::min<int64_t>(2048, std::max<int64_t>(1, (items + 255) / 256)));
    double* nxt = A2;
    for (int sweep = 0; sweep < MAX_SWEEPS && m > 1; ++sweep) {
      hipLaunchKernelGGL(jacobi_offnorm_kernel, dim3(1), dim3(1024), 0, stream, cur, m, lda,
                         norms);
      FD_LAUNCH_CHECK();
      double h[2] = {0.0, 0.0};
      FD_HIP_CHECK(hipMemcpyAsync(h, norms, sizeof(h), hipMemcpyDeviceToHost, stream));
      FD_HIP_CHECK(hipStreamSynchronize(stream));
      if (h[0] <= TOL * TOL * h[1]) break;
      for (int round = 0; round < me - 1; ++round) {
        hipLaunchKernelGGL(jacobi_round_kernel, dim3(grid), dim3(256), 0, stream, cur, nxt, lda,
                           Vw, m, me, round);
        FD_LAUNCH_CHECK();
        std::swap(cur, nxt);
      }
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
