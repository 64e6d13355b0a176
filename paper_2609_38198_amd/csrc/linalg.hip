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
// On the float64 matrix instruction v_mfma_f64_16x16x4f64 (operand A[i][k] on
// lane i + 16 k, B[k][j] on lane j + 16 k, result D[i][j] on lane
// j + 16 (i mod 4), register i / 4; i, j < 16, k < 4).  A wave owns a
// 64 x 16 NCB tile of C; its l-block q (q < 4) holds the rows l0 + 4 i + q of
// C and its c-block h (h < NCB) the columns c0 + NCB j + h, so that lane
// i + 16 k reads the four A values it needs from row k of a 4-row step with
// one 16-byte load and its NCB B values with one 4 NCB-byte load.  Products
// of float32 values are exact in float64 and the matrix unit sums them in
// float64.  The four waves of a workgroup take consecutive 16-row quarters of
// each 64 rows of the workgroup's chunk of rows and are added in LDS in a
// fixed order; the chunks' partial sums are then reduced in a fixed order.

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef double dbl4 __attribute__((ext_vector_type(4)));

constexpr int TN_ROWS = 64;   // rows of one workgroup iteration (4 waves x 4 steps x 4 rows)
constexpr int TN_WGS = 2048;  // workgroups aimed at (8 waves per SIMD)
constexpr int TN_CHUNKS_MIN = 32;
constexpr int TN_CHUNK_ROWS = 1024;

struct GemmTnShape {
  int ncb = 1, tiles_l = 1, tiles_c = 1;
  int64_t chunks = 1, rows_per_chunk = TN_ROWS;
};

static GemmTnShape gemm_tn_shape(int ma, int nb, int64_t N) {
  GemmTnShape g;
  g.ncb = nb <= 16 ? 1 : 2;
  g.tiles_l = (ma + 63) / 64;
  g.tiles_c = (nb + 16 * g.ncb - 1) / (16 * g.ncb);
  const int64_t tiles = int64_t(g.tiles_l) * g.tiles_c;
  // about TN_WGS workgroups of at least TN_ROWS rows each, but no more than
  // max(TN_CHUNKS_MIN, N / TN_CHUNK_ROWS) chunks (each chunk writes ma x nb
  // partial sums that the reduction reads back) and at most gemm_tn_chunks(N)
  // (the partial buffer's size)
  const int64_t want = std::min({gemm_tn_chunks(N), (TN_WGS + tiles - 1) / tiles,
                                 std::max<int64_t>(TN_CHUNKS_MIN, N / TN_CHUNK_ROWS)});
  g.rows_per_chunk = round_up((N + want - 1) / want, TN_ROWS);
  g.chunks = (N + g.rows_per_chunk - 1) / g.rows_per_chunk;
  return g;
}

// Loads of one 4-row step: row `row` of A (4 values) and of B (NCB values);
// with CLAMP rows at or past r1 read row r1 - 1 and give B the weight 0.
template <int NCB, bool VEC, bool CLAMP>
__device__ __forceinline__ void tn_load(const float* __restrict__ A, int64_t lda,
                                        const float* __restrict__ B, int64_t ldb, int64_t row,
                                        int64_t r1, const int (&lc)[4], const int (&cc)[NCB],
                                        float (&a)[4], float (&b)[NCB]) {
  const bool ok = !CLAMP || row < r1;
  const int64_t rc = CLAMP ? (ok ? row : r1 - 1) : row;
  const float* pa = A + rc * lda;
  const float* pb = B + rc * ldb;
  if constexpr (VEC) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(pa + lc[0]);
#pragma unroll
    for (int u = 0; u < 4; ++u) a[u] = v[u];
    if constexpr (NCB == 2) {
      const f32x2 w = *reinterpret_cast<const f32x2*>(pb + cc[0]);
      b[0] = ok ? w[0] : 0.f;
      b[1] = ok ? w[1] : 0.f;
    } else {
      b[0] = ok ? pb[cc[0]] : 0.f;
    }
  } else {
#pragma unroll
    for (int u = 0; u < 4; ++u) a[u] = pa[lc[u]];
#pragma unroll
    for (int h = 0; h < NCB; ++h) b[h] = ok ? pb[cc[h]] : 0.f;
  }
}

template <int NCB>
__device__ __forceinline__ void tn_mfma(const float (&a)[4], const float (&b)[NCB],
                                        dbl4 (&acc)[4][NCB]) {
  double bd[NCB];
#pragma unroll
  for (int h = 0; h < NCB; ++h) bd[h] = double(b[h]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const double ad = double(a[q]);
#pragma unroll
    for (int h = 0; h < NCB; ++h)
      acc[q][h] = __builtin_amdgcn_mfma_f64_16x16x4f64(ad, bd[h], acc[q][h], 0, 0, 0);
  }
}

// VEC: ma, lda multiples of 4, A 16-byte aligned and, for NCB = 2, nb, ldb
// even and B 8-byte aligned (the loads above are then vector loads).  Grid:
// tiles x chunks workgroups, numbered so that the workgroups on one XCD
// (blockIdx.x mod 8) take all tiles of consecutive chunks (B's rows stay in
// that XCD's L2).
template <int NCB, bool VEC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void gemm_tn_partial_kernel(
    const float* __restrict__ A, int64_t lda, int ma, const float* __restrict__ B, int64_t ldb,
    int nb, int64_t N, int64_t rows_per_chunk, int tiles_l, int tiles_c, int64_t total,
    double* __restrict__ part) {
  constexpr int E = 16 * NCB;  // result doubles per lane
  __shared__ double red[2][E * 64];
  const int64_t gid = blockIdx.x, per = total / 8, rem = total % 8, x = gid % 8;
  const int64_t lin = x * per + min(x, rem) + gid / 8;
  const int64_t tiles = int64_t(tiles_l) * tiles_c;
  const int64_t chunk = lin / tiles;
  const int tile = int(lin - chunk * tiles);
  const int l0 = 64 * (tile % tiles_l), c0 = 16 * NCB * (tile / tiles_l);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, k = lane >> 4;
  // columns past the edge read a valid column; their sums are not stored
  int lc[4], cc[NCB];
  if constexpr (VEC) {
    lc[0] = min(l0 + 4 * i, ma - 4);
    cc[0] = min(c0 + NCB * i, nb - NCB);
#pragma unroll
    for (int u = 1; u < 4; ++u) lc[u] = lc[0] + u;
#pragma unroll
    for (int h = 1; h < NCB; ++h) cc[h] = cc[0] + h;
  } else {
#pragma unroll
    for (int u = 0; u < 4; ++u) lc[u] = min(l0 + 4 * i + u, ma - 1);
#pragma unroll
    for (int h = 0; h < NCB; ++h) cc[h] = min(c0 + NCB * i + h, nb - 1);
  }
  const int64_t r0 = chunk * rows_per_chunk;
  const int64_t r1 = min(N, r0 + rows_per_chunk);
  dbl4 acc[4][NCB];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int h = 0; h < NCB; ++h) acc[q][h] = dbl4{0.0, 0.0, 0.0, 0.0};
  // this lane's row of step s of an iteration at r: r + 16 wave + 4 s + k
  const int64_t off = 16 * wave + k;
  int64_t r = r0;
  for (; r + TN_ROWS <= r1; r += TN_ROWS) {
    float a[4][4], b[4][NCB];
#pragma unroll
    for (int s = 0; s < 4; ++s)
      tn_load<NCB, VEC, false>(A, lda, B, ldb, r + off + 4 * s, r1, lc, cc, a[s], b[s]);
#pragma unroll
    for (int s = 0; s < 4; ++s) tn_mfma<NCB>(a[s], b[s], acc);
  }
  if (r < r1) {  // the ragged end of the last chunk
    float a[4][4], b[4][NCB];
#pragma unroll
    for (int s = 0; s < 4; ++s)
      tn_load<NCB, VEC, true>(A, lda, B, ldb, r + off + 4 * s, r1, lc, cc, a[s], b[s]);
#pragma unroll
    for (int s = 0; s < 4; ++s) tn_mfma<NCB>(a[s], b[s], acc);
  }
  // (wave 0 + wave 2) + (wave 1 + wave 3)
  if (wave >= 2) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int h = 0; h < NCB; ++h)
#pragma unroll
        for (int s = 0; s < 4; ++s) red[wave - 2][((q * NCB + h) * 4 + s) * 64 + lane] = acc[q][h][s];
  }
  __syncthreads();
  if (wave < 2) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int h = 0; h < NCB; ++h)
#pragma unroll
        for (int s = 0; s < 4; ++s) acc[q][h][s] += red[wave][((q * NCB + h) * 4 + s) * 64 + lane];
  }
  __syncthreads();
  if (wave == 1) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int h = 0; h < NCB; ++h)
#pragma unroll
        for (int s = 0; s < 4; ++s) red[0][((q * NCB + h) * 4 + s) * 64 + lane] = acc[q][h][s];
  }
  __syncthreads();
  if (wave != 0) return;
  double* out = part + chunk * int64_t(ma) * nb;
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int h = 0; h < NCB; ++h)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int l = l0 + 4 * (4 * s + k) + q, c = c0 + NCB * i + h;
        const double v = acc[q][h][s] + red[0][((q * NCB + h) * 4 + s) * 64 + lane];
        if (l < ma && c < nb) out[int64_t(l) * nb + c] = v;
      }
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
  const bool veca = ma % 4 == 0 && lda % 4 == 0 && reinterpret_cast<uintptr_t>(A) % 16 == 0;
  const bool vecb = g.ncb == 1 || (nb % 2 == 0 && ldb % 2 == 0 &&
                                   reinterpret_cast<uintptr_t>(B) % 8 == 0);
  const int64_t total = int64_t(g.tiles_l) * g.tiles_c * g.chunks;
  const dim3 grid{unsigned(total)};
#define FD_TN_LAUNCH(NCB, VEC)                                                                 \
  hipLaunchKernelGGL((gemm_tn_partial_kernel<NCB, VEC>), grid, dim3(256), 0, stream, A, lda, ma, B, \
                     ldb, nb, N, g.rows_per_chunk, g.tiles_l, g.tiles_c, total, part.p)
  if (g.ncb == 2) {
    if (veca && vecb) FD_TN_LAUNCH(2, true);
    else FD_TN_LAUNCH(2, false);
  } else {
    if (veca) FD_TN_LAUNCH(1, true);
    else FD_TN_LAUNCH(1, false);
  }
#undef FD_TN_LAUNCH
  FD_LAUNCH_CHECK();
  const int64_t count = int64_t(ma) * nb;
  hipLaunchKernelGGL(reduce_partials_kernel, dim3(nblk(count, 32)), dim3(256), 0, stream, part.p,
                     g.chunks, count, C, C32);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------ Z = beta Z + alpha Q C
// On the float32 matrix instruction v_mfma_f32_16x16x4f32 as Z^T = C^T Q^T:
// operand A = C^T[c][l] on lane c + 16 k, B = Q^T[l][row] on lane row + 16 k,
// result D[c][row] on lane row + 16 (c / 4), register c mod 4 (c, row < 16,
// k < 4).  A wave owns 16 MB rows x 16 NCB columns of Z.  In a group of 32
// values of l, lane x + 16 k takes l = L + 8 k + s at step s (s < 8): it reads
// its Q values of a row with two 16-byte loads and its C values with two
// 16-byte reads per column block from an LDS copy of C^T (staged NN_SL values
// of l at a time), and ends up holding 4 consecutive columns of each of its
// rows (one 16-byte store).  Sums are float32 in the matrix unit's order,
// the same on every run.

constexpr int NN_SL = 128;        // values of l per LDS slice of C
constexpr int NN_LD = NN_SL + 4;  // padded row of the LDS copy of C^T

// VEC: ma, ldq, nb, ldz multiples of 4 and Q, Z 16-byte aligned (vector loads
// of Q, vector loads and stores of Z).
template <int MB, int NCB, bool VEC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void gemm_nn_kernel(
    const float* __restrict__ Q, int64_t ldq, int ma, const float* __restrict__ C, int nb,
    float* __restrict__ Z, int64_t ldz, int64_t N, float alpha, float beta) {
  __shared__ __attribute__((aligned(16))) float ct[16 * NCB * NN_LD];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int x = lane & 15, k = lane >> 4;
  const int64_t rbase = (int64_t(blockIdx.x) * 4 + wave) * 16 * MB;
  // rows past N compute on row N - 1 and are not stored
  const float* qrow[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) qrow[mb] = Q + min(rbase + 16 * mb + x, N - 1) * ldq;
  f32x4 acc[MB][NCB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int h = 0; h < NCB; ++h) acc[mb][h] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int l0 = 0; l0 < ma; l0 += NN_SL) {
    const int len = min(NN_SL, ma - l0);
    __syncthreads();  // the previous slice is no longer read
    // C^T slice; l past ma and columns past nb hold 0 (so the clamped Q
    // values they meet add nothing)
    for (int e = threadIdx.x; e < NN_SL * 16 * NCB; e += 256) {
      const int l = e / (16 * NCB), c = e % (16 * NCB);
      ct[c * NN_LD + l] = (l < len && c < nb) ? C[int64_t(l0 + l) * nb + c] : 0.f;
    }
    __syncthreads();
    for (int L = 0; L < len; L += 32) {
      const int lq = l0 + L + 8 * k;  // this lane's first l of the group
      float a[MB][8], b[NCB][8];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        if constexpr (VEC) {
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            const int cs = lq + 4 * hf;
            const f32x4 v = *reinterpret_cast<const f32x4*>(qrow[mb] + (cs < ma ? cs : ma - 4));
#pragma unroll
            for (int u = 0; u < 4; ++u) a[mb][4 * hf + u] = v[u];
          }
        } else {
#pragma unroll
          for (int st = 0; st < 8; ++st) a[mb][st] = qrow[mb][min(lq + st, ma - 1)];
        }
      }
#pragma unroll
      for (int h = 0; h < NCB; ++h)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const f32x4 v =
              *reinterpret_cast<const f32x4*>(ct + (16 * h + x) * NN_LD + L + 8 * k + 4 * hf);
#pragma unroll
          for (int u = 0; u < 4; ++u) b[h][4 * hf + u] = v[u];
        }
#pragma unroll
      for (int st = 0; st < 8; ++st)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int h = 0; h < NCB; ++h)
            acc[mb][h] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[h][st], a[mb][st], acc[mb][h], 0, 0, 0);
    }
  }
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int64_t row = rbase + 16 * mb + x;
    if (row >= N) continue;
    float* zr = Z + row * ldz;
#pragma unroll
    for (int h = 0; h < NCB; ++h) {
      const int c0 = 16 * h + 4 * k;
      if constexpr (VEC) {
        if (c0 >= nb) continue;
        f32x4* z = reinterpret_cast<f32x4*>(zr + c0);
        f32x4 out;
        if (beta == 0.f) {
#pragma unroll
          for (int r = 0; r < 4; ++r) out[r] = alpha * acc[mb][h][r];
        } else {
          const f32x4 zo = *z;
#pragma unroll
          for (int r = 0; r < 4; ++r) out[r] = fmaf(beta, zo[r], alpha * acc[mb][h][r]);
        }
        *z = out;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (c0 + r < nb)
            zr[c0 + r] = (beta == 0.f) ? alpha * acc[mb][h][r]
                                       : fmaf(beta, zr[c0 + r], alpha * acc[mb][h][r]);
      }
    }
  }
}

void gemm_nn(const float* Q, int64_t ldq, int ma, const float* C, int nb, float* Z, int64_t ldz,
             int64_t N, float alpha, float beta, hipStream_t stream) {
  FD_REQUIRE(ma >= 1 && nb >= 1 && nb <= 64 && N >= 1, FD_ERR_INVALID_ARG,
             "internal: gemm_nn shape");
  const bool vec = ma % 4 == 0 && nb % 4 == 0 && ldq % 4 == 0 && ldz % 4 == 0 &&
                   reinterpret_cast<uintptr_t>(Q) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(Z) % 16 == 0;
  // 64 MB rows per workgroup: the most that still gives >= 1024 workgroups
  const int ncb = nb <= 16 ? 1 : nb <= 32 ? 2 : 4;
  const int mb = N >= 1024 * 256 ? 4 : N >= 1024 * 128 ? 2 : 1;
  const dim3 grid{nblk(N, 64 * mb)};
#define FD_NN_LAUNCH(MB, NCB)                                                                 \
  do {                                                                                        \
    if (vec)                                                                                  \
      hipLaunchKernelGGL((gemm_nn_kernel<MB, NCB, true>), grid, dim3(256), 0, stream, Q, ldq, \
                         ma, C, nb, Z, ldz, N, alpha, beta);                                  \
    else                                                                                      \
      hipLaunchKernelGGL((gemm_nn_kernel<MB, NCB, false>), grid, dim3(256), 0, stream, Q,     \
                         ldq, ma, C, nb, Z, ldz, N, alpha, beta);                             \
  } while (0)
  if (mb == 4 && ncb == 1) FD_NN_LAUNCH(4, 1);
  else if (mb == 4 && ncb == 2) FD_NN_LAUNCH(4, 2);
  else if (mb == 4) FD_NN_LAUNCH(4, 4);
  else if (mb == 2 && ncb == 1) FD_NN_LAUNCH(2, 1);
  else if (mb == 2 && ncb == 2) FD_NN_LAUNCH(2, 2);
  else if (mb == 2) FD_NN_LAUNCH(2, 4);
  else if (ncb == 1) FD_NN_LAUNCH(1, 1);
  else if (ncb == 2) FD_NN_LAUNCH(1, 2);
  else FD_NN_LAUNCH(1, 4);
#undef FD_NN_LAUNCH
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------ Cholesky + R^-1
// G (b x b, float64, row-major) = R^T R.  A column whose pivot falls below
// rel_tol times its own norm (numerically inside the span of the earlier
// columns), or whose norm is not positive, is flagged; it gets an identity
// row in R and is excluded from the later eliminations.  Output: Rinv
// (float32, upper triangular, ld b) and flags[b] (1 = replace this column).
// b <= B: one wave, lane t holds column t of the working matrix in
// registers (right-looking: step k turns entry k of every column into
// R[k][t] and updates the entries below it).  The pivot comes from lane k
// through v_readlane; row k of R is broadcast through LDS, and the reads of
// it are independent of each other.  Loops keep compile-time trip counts
// (steps k >= b see a zero column: flagged, unit pivot, no update) so the
// columns stay in registers.
__device__ __forceinline__ double readlane_d(double x, int lane) {
  const unsigned long long u = __double_as_longlong(x);
  const unsigned lo = unsigned(__builtin_amdgcn_readlane(int(unsigned(u)), lane));
  const unsigned hi = unsigned(__builtin_amdgcn_readlane(int(unsigned(u >> 32)), lane));
  return __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(hi) << 32) | lo));
}

template <int B>
__global__ __launch_bounds__(64) void chol_rinv_reg_kernel(const double* __restrict__ G, int b,
                                                           double rel_tol, float* __restrict__ Rinv,
                                                           int* __restrict__ flags) {
  constexpr int LD = B + 1;
  __shared__ double dgs[B], row[B], Rm[B * LD];
  const int t = threadIdx.x;
  const bool live = t < b;
  double a[B];
#pragma unroll
  for (int i = 0; i < B; ++i) a[i] = (live && i < b) ? G[i * b + t] : 0.0;
  if (t < B) dgs[t] = live ? G[t * b + t] : 0.0;
  __syncthreads();
  int fl = 0;
#pragma unroll
  for (int k = 0; k < B; ++k) {
    const double piv = readlane_d(a[k], k);
    const double d0 = dgs[k];
    const bool bad = !(d0 > 0.0) || !(piv > rel_tol * rel_tol * d0) || !isfinite(piv);
    const double rkk = bad ? 1.0 : sqrt(piv);
    if (t == k) fl = bad ? 1 : 0;
    // R[k][t]: the pivot on lane k, 0 left of it and in a flagged row
    const double r = t == k ? rkk : (t > k && !bad) ? a[k] / rkk : 0.0;
    a[k] = r;
    if (t < B) row[t] = r;
    __syncthreads();
#pragma unroll
    for (int i = k + 1; i < B; ++i) {
      const double rki = row[i];
      if (i <= t) a[i] = fma(-rki, r, a[i]);
    }
    __syncthreads();  // row is rewritten by the next step
  }
  if (t < B) {
#pragma unroll
    for (int i = 0; i < B; ++i) Rm[i * LD + t] = a[i];
  }
  __syncthreads();
  // Rinv: R X = I, lane t solves for column t (each solved entry removed
  // from the rows above it)
  double x[B];
#pragma unroll
  for (int i = 0; i < B; ++i) x[i] = i == t ? 1.0 : 0.0;
#pragma unroll
  for (int l = B - 1; l >= 0; --l) {
    x[l] = x[l] / Rm[l * LD + l];
#pragma unroll
    for (int i = 0; i < l; ++i) x[i] = fma(-Rm[i * LD + l], x[l], x[i]);
  }
  if (live) {
#pragma unroll
    for (int i = 0; i < B; ++i)
      if (i < b) Rinv[i * b + t] = float(x[i]);
    flags[t] = fl;
  }
}

// 32 < b <= 64: the same steps with the working matrix in LDS (thread t owns
// column t; step k writes row k of R, then every thread updates its column).
__global__ __launch_bounds__(64) void chol_rinv_kernel(const double* __restrict__ G, int b,
                                                       double rel_tol, float* __restrict__ Rinv,
                                                       int* __restrict__ flags) {
  constexpr int LD = 65;  // padded rows: a column of the matrix sits in 64 banks
  __shared__ double A[64 * LD];
  __shared__ double R[64 * LD];
  __shared__ double X[64 * LD];
  __shared__ double dg[64];
  __shared__ int flag[64];
  const int t = threadIdx.x;
  for (int e = t; e < 64 * LD; e += 64) {
    const int i = e / LD, j = e % LD;
    A[e] = (i < b && j < b) ? G[i * b + j] : 0.0;
    R[e] = 0.0;
    X[e] = 0.0;
  }
  dg[t] = t < b ? G[t * b + t] : 0.0;
  __syncthreads();
  for (int k = 0; k < b; ++k) {
    const double diag = dg[k];
    const double piv = A[k * LD + k];
    const bool bad = !(diag > 0.0) || !(piv > rel_tol * rel_tol * diag) || !isfinite(piv);
    const double rkk = bad ? 1.0 : sqrt(piv);
    const bool mine = t > k && t < b;
    const double r = (mine && !bad) ? A[k * LD + t] / rkk : 0.0;
    if (mine) R[k * LD + t] = r;
    if (t == k) {
      R[k * LD + k] = rkk;
      flag[k] = bad ? 1 : 0;
    }
    __syncthreads();
    if (mine)
      for (int i = k + 1; i <= t; ++i) A[i * LD + t] -= R[k * LD + i] * r;
    __syncthreads();
  }
  if (t < b) {
    X[t * LD + t] = 1.0;
    for (int l = t; l >= 0; --l) {
      const double xl = X[l * LD + t] / R[l * LD + l];
      X[l * LD + t] = xl;
      for (int i = 0; i < l; ++i) X[i * LD + t] -= R[i * LD + l] * xl;
    }
  }
  __syncthreads();
  for (int e = t; e < b * b; e += 64) Rinv[e] = float(X[(e / b) * LD + e % b]);
  if (t < b) flags[t] = flag[t];
}

void chol_rinv(const double* G, int b, double rel_tol, float* Rinv, int* flags,
               hipStream_t stream) {
  FD_REQUIRE(b >= 1 && b <= 64, FD_ERR_INVALID_ARG, "internal: chol size");
  if (b <= 16)
    hipLaunchKernelGGL(chol_rinv_reg_kernel<16>, dim3(1), dim3(64), 0, stream, G, b, rel_tol,
                       Rinv, flags);
  else if (b <= 32)
    hipLaunchKernelGGL(chol_rinv_reg_kernel<32>, dim3(1), dim3(64), 0, stream, G, b, rel_tol,
                       Rinv, flags);
  else
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
// R_i^T X R_j.  Two ways to run the sweeps:
//   * m <= JL_MAX: one workgroup holds the upper triangle in LDS and runs
//     whole sweeps with a barrier between rounds (jacobi_lds_kernel); the
//     rotations are logged and replayed on the eigenvector matrix by a
//     second kernel (jacobi_replay_kernel);
//   * larger m: block Jacobi (the block-cyclic orderings of Golub & Van Loan,
//     Sec. 8.5.5).  The indices form blocks of BJ_S; a round pairs the blocks
//     by the circle method, each pair of blocks (2 BJ_S indices) gets
//     rotations on its principal submatrix in LDS, and their product U_u
//     then acts on A tile by tile, A_uv <- U_u^T A_uv U_v, and on the
//     eigenvector matrix, V_:v <- V_:v U_v.  On the first round of a sweep
//     the submatrix gets one cyclic sweep (the pairs inside each block), on
//     the others only its cross-block pairs: every pair of indices meets once
//     per sweep.  One launch per round (bj_round_kernel) applies round r and
//     solves round r + 1 side by side (A double-buffered); a sweep takes
//     m / BJ_S - 1 launches instead of m - 1; A is first made exactly
//     symmetric from its upper triangle (the submatrix builds read tiles
//     through their transposes).  After each sweep the
//     off-diagonal Frobenius norm is checked on the host (one pair of
//     scalars read back).
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

// rotation (c, s) annihilating A_pq: t = tan of the angle is the smaller
// root of t^2 + 2 tau t - 1 = 0, tau = (aqq - app) / (2 apq) (the 2 x 2
// symmetric Schur decomposition of Golub & Van Loan).  With d = aqq - app,
// r = sqrt(d^2 + 4 apq^2) and e = |d| + r, t = sign(d) 2 apq / e, so (c, s)
// is the unit vector along (e, sign(d) 2 apq), normalised as a vector
// (1 / |(e, 2 apq)|, which keeps c^2 + s^2 = 1 to float64 rounding): one
// square root and one reciprocal square root on the dependent path, no
// division.
__device__ __forceinline__ void jacobi_rotation(double app, double aqq, double apq, double& c,
                                                double& s) {
  const double d = aqq - app;
  const double a2 = 2.0 * apq;
  const double r = sqrt(fma(d, d, a2 * a2));
  const double e = fabs(d) + r;
  const double q = rsqrt(fma(e, e, a2 * a2));
  c = e * q;
  s = (d >= 0.0 ? a2 : -a2) * q;
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

__global__ void jacobi_init_kernel(double* __restrict__ V, int m) {
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e < int64_t(m) * m) V[e] = (e / m == e % m) ? 1.0 : 0.0;
}

// whether diagonal entry (dj, j) sorts before (di, i): descending, ties by
// index, NaN after every number (ties among NaNs by index).  A strict total
// order for any input, so the ranks below always form a permutation.
__device__ __forceinline__ bool sorts_before(double dj, int j, double di, int i) {
  const bool nj = dj != dj, ni = di != di;
  if (nj || ni) return !nj || (ni && j < i);
  return dj > di || (dj == di && j < i);
}

// theta = diag(A) sorted descending, perm[rank] = the index of that rank;
// every workgroup stages the diagonal (m <= 1024) in LDS
__global__ __launch_bounds__(256) void jacobi_rank_kernel(const double* __restrict__ A, int m,
                                                          int lda, double* __restrict__ theta,
                                                          int* __restrict__ perm) {
  __shared__ double dg[1024];
  for (int j = threadIdx.x; j < m; j += 256) dg[j] = A[int64_t(j) * lda + j];
  __syncthreads();
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  const double di = dg[i];
  int rank = 0;
  for (int j = 0; j < m; ++j) rank += (j != i && sorts_before(dg[j], j, di, i)) ? 1 : 0;
  theta[rank] = di;
  perm[rank] = i;
}

// S[r][k] = V[r][perm[k]]: the columns of V in rank order (perm is a
// permutation of 0 .. m - 1 by construction; the clamp keeps the gather in
// range whatever it holds)
__global__ __launch_bounds__(256) void jacobi_permute_kernel(const double* __restrict__ V, int m,
                                                             const int* __restrict__ perm,
                                                             double* __restrict__ S, int lds) {
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= int64_t(m) * m) return;
  const int r = int(e / m), k = int(e % m);
  const int src = int(min(unsigned(perm[k]), unsigned(m - 1)));
  S[int64_t(r) * lds + k] = V[int64_t(r) * m + src];
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
// ---- block Jacobi for JL_MAX < m <= 1024 (the scheme in the header above)
constexpr int BJ_S = 16;          // indices per block
constexpr int BJ_W = 2 * BJ_S;    // indices per pair of blocks
constexpr int BJ_LD = BJ_W + 1;   // LDS row stride of a BJ_W x BJ_W matrix
constexpr int BJ_PART = 64;       // workgroups of the off-diagonal norm

// blocks (an even count: a padding block when needed) for an m x m matrix
static inline int bj_blocks(int m) {
  const int nb = (m + BJ_S - 1) / BJ_S;
  return nb + (nb & 1);
}

// scratch of the block path: the U_u (BJ_W^2 each) and moved flags of two
// consecutive rounds, and the partial norms (per workgroup of the first
// check, per tile of A after)
static inline size_t bj_doubles(int m) {
  const int P = bj_blocks(m) / 2;
  return 2 * (size_t(P) * BJ_W * BJ_W + P) + 2 * std::max(BJ_PART, P * (P + 1) / 2);
}

// scratch that every size up to m needs
size_t jacobi_log_doubles(int m) {
  const int mc = std::min(m, JL_MAX);
  const int me = mc + (mc & 1);
  const size_t lds_path = size_t(JL_SWEEPS) * me * std::max(me - 1, 1);
  return m > JL_MAX ? std::max(lds_path, bj_doubles(m)) : lds_path;
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


// global index of local index l of the pair of blocks (bp, bq); >= m marks
// padding (a zero row and column: its rotations are the identity)
__device__ __forceinline__ int bj_global(int bp, int bq, int l) {
  return l < BJ_S ? bp * BJ_S + l : bq * BJ_S + (l - BJ_S);
}

// rotation (c, s) annihilating the entry apq of a symmetric matrix with
// diagonal entries app, aqq; the identity when apq is zero or negligible next
// to both in float64 (100 |apq| vanishes when added to either, Rutishauser's
// rule).  Branch-free: the rotation is always formed (a zero d and apq give
// NaNs there) and the identity selected.
__device__ __forceinline__ double2 bj_rotation(double app, double aqq, double apq) {
  double c, sn;
  jacobi_rotation(app, aqq, apq, c, sn);
  const double g = 100.0 * fabs(apq);
  const bool skip = fabs(app) + g == fabs(app) && fabs(aqq) + g == fabs(aqq);  // also apq = 0
  return skip ? make_double2(1.0, 0.0) : make_double2(c, sn);
}

// x if keep, else +0.0, by a bit mask: no select, so the load that produced x
// is not moved behind a branch
__device__ __forceinline__ double masked(double x, bool keep) {
  return __longlong_as_double(__double_as_longlong(x) & (keep ? -1LL : 0LL));
}

// x of lane (l + 1) mod 16 of this lane's 16-lane row (DPP row rotate)
__device__ __forceinline__ double row_next(double x) {
  constexpr int ROW_ROR_15 = 0x12F;
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(x), ROW_ROR_15, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(x), ROW_ROR_15, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}

// One inner round on the BJ_W x BJ_W submatrix Sc -> Sn and the rotation
// product Jm, for thread (ti, tj) with pairs (pi, qi) = pair ti and
// (pj, qj) = pair tj of the round.  Every LDS read comes first (the entries of
// rotation tj, the 2 x 2 block rows pi, qi x columns pj, qj, the entries of J
// on rows ti, ti + 16 and columns pj, qj); rotation tj is formed on this lane
// and rotation ti fetched from lane ti of the 16-lane row (whose tj is ti).
// Returns whether rotation tj is not the identity.
__device__ __forceinline__ bool bj_inner_round(const double* __restrict__ Sc,
                                               double* __restrict__ Sn, double* __restrict__ Jm,
                                               int ti, int pi, int qi, int pj, int qj) {
  const double jpp = Sc[pj * BJ_LD + pj], jqq = Sc[qj * BJ_LD + qj], jpq = Sc[pj * BJ_LD + qj];
  const double a = Sc[pi * BJ_LD + pj], b = Sc[pi * BJ_LD + qj];
  const double d = Sc[qi * BJ_LD + pj], e = Sc[qi * BJ_LD + qj];
  double jp[2], jq[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    jp[h] = Jm[(ti + 16 * h) * BJ_LD + pj];
    jq[h] = Jm[(ti + 16 * h) * BJ_LD + qj];
  }
  const double2 rj = bj_rotation(jpp, jqq, jpq);
  const double2 ri = make_double2(__shfl(rj.x, ti, 16), __shfl(rj.y, ti, 16));
  // block (ti, tj) becomes R_i^T X R_j
  const double a1 = ri.x * a - ri.y * d, b1 = ri.x * b - ri.y * e;
  const double d1 = ri.y * a + ri.x * d, e1 = ri.y * b + ri.x * e;
  Sn[pi * BJ_LD + pj] = rj.x * a1 - rj.y * b1;
  Sn[pi * BJ_LD + qj] = rj.y * a1 + rj.x * b1;
  Sn[qi * BJ_LD + pj] = rj.x * d1 - rj.y * e1;
  Sn[qi * BJ_LD + qj] = rj.y * d1 + rj.x * e1;
  // columns pj, qj of J (the identity rotation rewrites them unchanged)
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    Jm[(ti + 16 * h) * BJ_LD + pj] = rj.x * jp[h] - rj.y * jq[h];
    Jm[(ti + 16 * h) * BJ_LD + qj] = rj.y * jp[h] + rj.x * jq[h];
  }
  return rj.y != 0.0;
}

constexpr int BJ_TILE = BJ_W * BJ_LD;  // doubles of one padded BJ_W x BJ_W matrix in LDS

// float64 matrix instruction v_mfma_f64_16x16x4f64 (lane layouts as in C = A^T B above)

// One launch per round of the block Jacobi.  Workgroups [0, nsolve) take the
// pairs of blocks of round rs: each builds its BJ_W x BJ_W principal
// submatrix of the current A, runs its rotations (one cyclic sweep on round 0
// of a sweep, the cross-block pairs otherwise; one barrier per inner round,
// the submatrix double-buffered in LDS and every thread forming the two
// rotations it needs), and writes their product U_u and a moved flag to
// Us, fs.  The others apply round ra (rotations Ua, flags fa): tiles (u, v),
// u <= v, of A0 become U_u^T A0_uv U_v in A1 (mirrored: A1 is exactly
// symmetric), and the tiles of V (BJ_W rows x the columns of pair v) become
// V_:v U_v in place.
//
// The current A is A1 of this launch's apply, which is not written yet: a
// solve of round rs = ra + 1 forms its submatrix from A0 and Ua itself (its
// two blocks sat in two different pairs of round ra; each quadrant is
// U_ui[:, half]^T A0_{ui uj} U_uj[:, half]).  With ra < 0 (the first launch)
// A0 is the current matrix.  With part != null the apply workgroups of A
// write the squared off-diagonal and total norms of their tiles of A1 to
// part[2 w], part[2 w + 1] (w = tile index).  Workgroups of 256 threads: in
// the inner rounds thread (i, j) = (t / 16, t % 16); the submatrix build and
// the apply run on float64 matrix instructions, one 16 x 16 block per wave.
__global__ __launch_bounds__(256) void bj_round_kernel(
    const double* __restrict__ A0, double* __restrict__ A1, double* __restrict__ V, int lda,
    int m, int nbk, int ra, const double* __restrict__ Ua, const double* __restrict__ fa, int rs,
    double* __restrict__ Us, double* __restrict__ fs, int nsolve, int ntile_a,
    double* __restrict__ part) {
  __shared__ double L[3 * BJ_TILE];
  __shared__ int2 owner[64];  // block -> (pair, half) in round ra
  __shared__ int2 pairs[32];  // pair -> its two blocks in round ra
  __shared__ int moved;
  const int P = nbk / 2;
  const int t = threadIdx.x;
  const int ti = t >> 4, tj = t & 15;
  static_assert(BJ_S == 16 && BJ_W == 32, "thread (i, j) owns one 2 x 2 block per inner round");

  if (int(blockIdx.x) < nsolve) {
    // ------------------------------------------------------------ solve
    const int u = blockIdx.x;
    int bp, bq;
    circle_pair(nbk, rs, u, bp, bq);
    double* S0 = L;
    double* S1 = L + BJ_TILE;
    double* Jm = L + 2 * BJ_TILE;
    if (ra < 0) {
      constexpr int NL = BJ_W * BJ_W / 256;
      double sr[NL];
#pragma unroll
      for (int k = 0; k < NL; ++k) {
        const int e = t + 256 * k;
        const int gi = bj_global(bp, bq, e / BJ_W), gj = bj_global(bp, bq, e % BJ_W);
        sr[k] = (gi < m && gj < m) ? A0[int64_t(gi) * lda + gj] : 0.0;
      }
#pragma unroll
      for (int k = 0; k < NL; ++k) {
        const int e = t + 256 * k;
        S0[(e / BJ_W) * BJ_LD + e % BJ_W] = sr[k];
      }
    } else {
      if (t < P) {
        int p, q;
        circle_pair(nbk, ra, t, p, q);
        owner[p] = make_int2(t, 0);
        owner[q] = make_int2(t, 1);
        pairs[t] = make_int2(p, q);
      }
      __syncthreads();
      const int2 o1 = owner[bp], o2 = owner[bq];
      const int wv = t >> 6, l = t & 63, li = l & 15, lk = l >> 4;
      if (wv < 3) {
        // quadrant (qa, qb) of the new submatrix (blocks qa ? bq : bp and
        // qb ? bq : bp), one wave each: Y = X Jj[:, cj .. cj + 15] with X the
        // old tile of the two pairs, then Z = Ji[:, ci .. ci + 15]^T Y, on
        // float64 matrix instructions
        const int qa = wv == 2 ? 1 : 0, qb = wv == 0 ? 0 : 1;
        const int2 oa = qa ? o2 : o1, ob = qb ? o2 : o1;
        const int2 pa = pairs[oa.x], pb = pairs[ob.x];
        const double* Ji = Ua + int64_t(oa.x) * BJ_W * BJ_W + 16 * oa.y;
        const double* Jj = Ua + int64_t(ob.x) * BJ_W * BJ_W + 16 * ob.y;
        // every operand load in flight at once, none behind a branch: padding
        // rows and columns (index >= m) read a clamped in-range entry and are
        // zeroed (32-bit offsets: m, lda <= 1024).  A0 is exactly symmetric,
        // so X[16 h + i][4 s + k] is read as A0[col 4 s + k][row 16 h + i]:
        // the 16 lanes of a k read 16 consecutive doubles, and a load touches
        // four 128-byte lines instead of sixteen partly used ones
        double xa[2][8], jb[8], ja[8];
        int co[2];
        bool cv[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int gr = bj_global(pa.x, pa.y, 16 * h + li);
          cv[h] = gr < m;
          co[h] = min(gr, m - 1);
        }
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const int gc = bj_global(pb.x, pb.y, 4 * s + lk);
          const int ro = int(__umul24(unsigned(min(gc, m - 1)), unsigned(lda)));
#pragma unroll
          for (int h = 0; h < 2; ++h) xa[h][s] = masked(A0[ro + co[h]], cv[h] && gc < m);
          jb[s] = Jj[(4 * s + lk) * BJ_W + li];
          ja[s] = Ji[(4 * s + lk) * BJ_W + li];
        }
        __builtin_amdgcn_sched_barrier(0);  // all loads issued before the first wait
        dbl4 y0 = {0.0, 0.0, 0.0, 0.0}, y1 = y0;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          y0 = __builtin_amdgcn_mfma_f64_16x16x4f64(xa[0][s], jb[s], y0, 0, 0, 0);
          y1 = __builtin_amdgcn_mfma_f64_16x16x4f64(xa[1][s], jb[s], y1, 0, 0, 0);
        }
        // the result layout is the B operand layout of the next product: lane
        // j + 16 k holds Y[4 s + k][j] in register s of y0 (s < 4), y1 (s >= 4)
        dbl4 z0 = {0.0, 0.0, 0.0, 0.0}, z1 = z0;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          z0 = __builtin_amdgcn_mfma_f64_16x16x4f64(ja[s], y0[s], z0, 0, 0, 0);
          z1 = __builtin_amdgcn_mfma_f64_16x16x4f64(ja[s + 4], y1[s], z1, 0, 0, 0);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const double z = z0[r] + z1[r];
          const int i = lk + 4 * r;
          S0[(16 * qa + i) * BJ_LD + 16 * qb + li] = z;
          if (qa != qb) S0[(16 * qb + li) * BJ_LD + 16 * qa + i] = z;
        }
      }
    }
    for (int e = t; e < BJ_W * BJ_W; e += 256)
      Jm[(e / BJ_W) * BJ_LD + e % BJ_W] = (e / BJ_W == e % BJ_W) ? 1.0 : 0.0;
    if (t == 0) moved = 0;
    __syncthreads();
    bool mv = false;
    if (rs == 0) {
      // one cyclic sweep over all pairs of the submatrix
      double* Sc = S0;
      double* Sn = S1;
      for (int r = 0; r < BJ_W - 1; ++r) {
        int pi, qi, pj, qj;
        circle_pair(BJ_W, r, ti, pi, qi);
        circle_pair(BJ_W, r, tj, pj, qj);
        mv |= bj_inner_round(Sc, Sn, Jm, ti, pi, qi, pj, qj);
        __syncthreads();
        double* tmp = Sc;
        Sc = Sn;
        Sn = tmp;
      }
    } else {
      // the pairs across the two blocks: local index k meets q(k) =
      // BJ_S + (k + r) mod BJ_S in inner round r.  Thread (ti, tj) keeps
      // a = S[ti][tj], b = S[ti][q(tj)] and J[ti + 16 h][tj], J[ti + 16 h][q(tj)]
      // in registers (J = I at the start); as q(tj) of the next round is
      // q(tj + 1) of this one, b and the q-column of J pass to the next lane of
      // the 16-lane row after each round.  LDS keeps the whole submatrix for
      // the rotations' entries and the entries d = S[q(ti)][tj], e =
      // S[q(ti)][q(tj)] (written by other rows).
      double a = S0[ti * BJ_LD + tj], b = S0[ti * BJ_LD + BJ_S + tj];
      double jp[2] = {ti == tj ? 1.0 : 0.0, 0.0}, jq[2] = {0.0, ti == tj ? 1.0 : 0.0};
#pragma unroll 2
      for (int r = 0; r < BJ_S; ++r) {
        const double* Sc = (r & 1) ? S1 : S0;
        double* Sn = (r & 1) ? S0 : S1;
        const int qi = BJ_S + ((ti + r) & (BJ_S - 1)), qj = BJ_S + ((tj + r) & (BJ_S - 1));
        const double app = Sc[tj * BJ_LD + tj], aqq = Sc[qj * BJ_LD + qj];
        const double apq = Sc[tj * BJ_LD + qj];
        const double d = Sc[qi * BJ_LD + tj], e = Sc[qi * BJ_LD + qj];
        const double2 rj = bj_rotation(app, aqq, apq);
        const double2 ri = make_double2(__shfl(rj.x, ti, 16), __shfl(rj.y, ti, 16));
        const double a1 = ri.x * a - ri.y * d, b1 = ri.x * b - ri.y * e;
        const double d1 = ri.y * a + ri.x * d, e1 = ri.y * b + ri.x * e;
        a = rj.x * a1 - rj.y * b1;
        b = rj.y * a1 + rj.x * b1;
        Sn[ti * BJ_LD + tj] = a;
        Sn[ti * BJ_LD + qj] = b;
        Sn[qi * BJ_LD + tj] = rj.x * d1 - rj.y * e1;
        Sn[qi * BJ_LD + qj] = rj.y * d1 + rj.x * e1;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const double jn = rj.x * jp[h] - rj.y * jq[h];
          jq[h] = row_next(rj.y * jp[h] + rj.x * jq[h]);
          jp[h] = jn;
        }
        b = row_next(b);
        mv |= rj.y != 0.0;
        __syncthreads();
      }
      // after BJ_S rounds q(tj) = BJ_S + tj again
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        Jm[(ti + 16 * h) * BJ_LD + tj] = jp[h];
        Jm[(ti + 16 * h) * BJ_LD + BJ_S + tj] = jq[h];
      }
    }
    if (ti == tj && mv) moved = 1;  // every writer stores the same value
    __syncthreads();
    double* Uo = Us + int64_t(u) * BJ_W * BJ_W;
    for (int e = t; e < BJ_W * BJ_W; e += 256) Uo[e] = Jm[(e / BJ_W) * BJ_LD + e % BJ_W];
    if (t == 0) fs[u] = moved ? 1.0 : 0.0;
    return;
  }

  // -------------------------------------------------------------- apply
  const int w = blockIdx.x - nsolve;
  const bool on_a = w < ntile_a;
  int u = 0, v = 0, rc = 0;
  if (on_a) {
    int rem = w;
    while (rem >= P - u) {
      rem -= P - u;
      ++u;
    }
    v = u + rem;
  } else {
    rc = (w - ntile_a) / P;
    v = (w - ntile_a) % P;
  }
  const bool moved_u = on_a && fa[u] != 0.0, moved_v = fa[v] != 0.0;
  // V tiles in place: nothing to do for an unrotated pair (uniform per workgroup)
  if (!on_a && !moved_v) return;
  int bpu = 0, bqu = 0, bpv, bqv;
  circle_pair(nbk, ra, v, bpv, bqv);
  if (on_a) circle_pair(nbk, ra, u, bpu, bqu);
  // wave (a, c) of the workgroup forms the 16 x 16 block (rows 16 a .., columns
  // 16 c ..) of each stage on float64 matrix instructions; stage 1 puts
  // Y = U_u^T X (a tile of A whose row pair u rotated) or Y = X into LDS, stage
  // 2 takes Z = Y U_v (column pair v rotated) or Z = Y
  const int wv = t >> 6, l = t & 63, li = l & 15, lk = l >> 4;
  const int a = wv >> 1, c = wv & 1;
  // this lane's column of X in both stages is 16 c + li; loads are clamped
  // into the matrix and padding zeroed, so none sits behind a branch
  const int gjl = bj_global(bpv, bqv, 16 * c + li);
  const int gjc = min(gjl, m - 1);
  const double* xb_ = on_a ? A0 : V;
  const unsigned xld = unsigned(on_a ? lda : m);
  auto xval = [&](int i) -> double {
    const int row = on_a ? bj_global(bpu, bqu, i) : rc * BJ_W + i;
    return masked(xb_[int(__umul24(unsigned(min(row, m - 1)), xld)) + gjc], row < m && gjl < m);
  };
  double* Y = L;
  {
    dbl4 y = {0.0, 0.0, 0.0, 0.0};
    if (on_a && moved_u) {
      const double* Uu = Ua + int64_t(u) * BJ_W * BJ_W;
      double ua[8], xb[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        ua[s] = Uu[(4 * s + lk) * BJ_W + 16 * a + li];  // A[i][k] = U_u[4 s + k][16 a + i]
        xb[s] = xval(4 * s + lk);                       // B[k][j] = X[4 s + k][16 c + j]
      }
      __builtin_amdgcn_sched_barrier(0);  // all loads issued before the first wait
#pragma unroll
      for (int s = 0; s < 8; ++s) y = __builtin_amdgcn_mfma_f64_16x16x4f64(ua[s], xb[s], y, 0, 0, 0);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) y[r] = xval(16 * a + lk + 4 * r);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) Y[(16 * a + lk + 4 * r) * BJ_LD + 16 * c + li] = y[r];
  }
  __syncthreads();
  dbl4 z;
  if (moved_v) {
    const double* Uv = Ua + int64_t(v) * BJ_W * BJ_W;
    double ya[8], vb[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      ya[s] = Y[(16 * a + li) * BJ_LD + 4 * s + lk];  // A[i][k] = Y[16 a + i][4 s + k]
      vb[s] = Uv[(4 * s + lk) * BJ_W + 16 * c + li];  // B[k][j] = U_v[4 s + k][16 c + j]
    }
    __builtin_amdgcn_sched_barrier(0);  // all loads issued before the first wait
    dbl4 z0 = {0.0, 0.0, 0.0, 0.0}, z1 = z0;
#pragma unroll
    for (int s = 0; s < 8; s += 2) {
      z0 = __builtin_amdgcn_mfma_f64_16x16x4f64(ya[s], vb[s], z0, 0, 0, 0);
      z1 = __builtin_amdgcn_mfma_f64_16x16x4f64(ya[s + 1], vb[s + 1], z1, 0, 0, 0);
    }
    z = z0 + z1;
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) z[r] = Y[(16 * a + lk + 4 * r) * BJ_LD + 16 * c + li];
  }
  double off = 0.0, all = 0.0;
  const int j = 16 * c + li;
  const int gj = bj_global(bpv, bqv, j);
  if (gj < m) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * a + lk + 4 * r;
      const double val = z[r];
      if (on_a) {
        const int gi = bj_global(bpu, bqu, i);
        if (gi >= m || (u == v && i > j)) continue;
        A1[int64_t(gi) * lda + gj] = val;
        A1[int64_t(gj) * lda + gi] = val;
        const double sq = val * val;
        if (gi == gj) {
          all += sq;
        } else {
          off += 2.0 * sq;
          all += 2.0 * sq;
        }
      } else {
        const int row = rc * BJ_W + i;
        if (row < m) V[int64_t(row) * m + gj] = val;
      }
    }
  }
  if (part != nullptr && on_a) {
    // fixed-order tree over the workgroup, in LDS no thread reads any more
    __syncthreads();
    double* r0 = L;
    double* r1 = L + 256;
    r0[t] = off;
    r1[t] = all;
    __syncthreads();
    for (int s2 = 128; s2 > 0; s2 >>= 1) {
      if (t < s2) {
        r0[t] += r0[t + s2];
        r1[t] += r1[t + s2];
      }
      __syncthreads();
    }
    if (t == 0) {
      part[2 * w] = r0[0];
      part[2 * w + 1] = r1[0];
    }
  }
}

// A[r][c] = A[c][r] for r > c: A exactly symmetric, from its upper triangle
__global__ void symmetrize_kernel(double* __restrict__ A, int m, int lda) {
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= int64_t(m) * m) return;
  const int r = int(e / m), c = int(e % m);
  if (r > c) A[int64_t(r) * lda + c] = A[int64_t(c) * lda + r];
}

// part[2 b], part[2 b + 1] = squared off-diagonal and total Frobenius norms of
// rows b, b + BJ_PART, ... (fixed order); out = the sums of the parts in order
__global__ __launch_bounds__(256) void offnorm_partial_kernel(const double* __restrict__ A, int m,
                                                              int lda, double* __restrict__ part) {
  __shared__ double r0[256], r1[256];
  const int t = threadIdx.x;
  double off = 0.0, all = 0.0;
  for (int i = blockIdx.x; i < m; i += gridDim.x)
    for (int j = t; j < m; j += blockDim.x) {
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
    part[2 * blockIdx.x] = r0[0];
    part[2 * blockIdx.x + 1] = r1[0];
  }
}

__global__ __launch_bounds__(256) void offnorm_finish_kernel(const double* __restrict__ part,
                                                             int nparts,
                                                             double* __restrict__ out) {
  __shared__ double r0[256], r1[256];
  const int t = threadIdx.x;
  double off = 0.0, all = 0.0;
  for (int b = t; b < nparts; b += blockDim.x) {
    off += part[2 * b];
    all += part[2 * b + 1];
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

int jacobi_eig(double* A, double* A2, int m, int lda, double* Vw, double* theta, double* S,
               int lds, double* norms, FSpanD log, int* state, hipStream_t stream) {
  FD_REQUIRE(m >= 1 && m <= 1024, FD_ERR_UNSUPPORTED, "projected matrix larger than 1024");
  constexpr int MAX_SWEEPS = 60;
  constexpr double TOL = 1e-13;
  hipLaunchKernelGGL(jacobi_init_kernel, dim3(nblk(int64_t(m) * m, 256)), dim3(256), 0, stream, Vw,
                     m);
  FD_LAUNCH_CHECK();
  int sweeps = 0;
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
      sweeps += h[0] / std::max(m + (m & 1) - 1, 1);
      if (h[1]) break;
    }
  } else if (m > 1) {
    FD_REQUIRE(lda >= m && A2 != nullptr, FD_ERR_INVALID_ARG, "internal: block jacobi buffers");
    // Stop at off(A) <= 1e-10 |A|_F.  A Ritz pair (theta_i, S e_i) of T then
    // has residual |T s - theta s| <= off(A), about 3e-9 for the Markov
    // operators here (|T|_F <= sqrt(m)), and theta_i moves by no more; the
    // solver accepts pairs only on their explicitly computed residuals
    // |W s - theta Q s| (tolerance 1e-5), and the kept block of T is
    // re-projected at every restart, so the last sweeps of a 1e-13 stop
    // (one or two of about eight) bought nothing the caller sees.
    constexpr double TOL_BLOCK = 1e-10;
    check_span_d(log, bj_doubles(m), "block jacobi scratch");
    const int nbk = bj_blocks(m), P = nbk / 2;
    // a solve of round r + 1 sits in another pair than in round r only when a
    // sweep has more than one round
    FD_REQUIRE(nbk >= 4, FD_ERR_INVALID_ARG, "internal: block jacobi needs two rounds per sweep");
    const int ntile_a = P * (P + 1) / 2;
    const int ntile_v = ((m + BJ_W - 1) / BJ_W) * P;
    double* U[2] = {log.p, log.p + size_t(P) * BJ_W * BJ_W};
    double* F[2] = {U[1] + size_t(P) * BJ_W * BJ_W, U[1] + size_t(P) * BJ_W * BJ_W + P};
    double* part = F[1] + P;
    double* nxt = A2;
    // the submatrix builds read A through its transpose
    hipLaunchKernelGGL(symmetrize_kernel, dim3(nblk(int64_t(m) * m, 256)), dim3(256), 0, stream, A,
                       m, lda);
    FD_LAUNCH_CHECK();
    auto check = [&](int nparts) {
      hipLaunchKernelGGL(offnorm_finish_kernel, dim3(1), dim3(256), 0, stream, part, nparts,
                         norms);
      FD_LAUNCH_CHECK();
      double h[2] = {0.0, 0.0};
      FD_HIP_CHECK(hipMemcpyAsync(h, norms, sizeof(h), hipMemcpyDeviceToHost, stream));
      FD_HIP_CHECK(hipStreamSynchronize(stream));
      return h[0] <= TOL_BLOCK * TOL_BLOCK * h[1];
    };
    hipLaunchKernelGGL(offnorm_partial_kernel, dim3(BJ_PART), dim3(256), 0, stream, cur, m, lda,
                       part);
    FD_LAUNCH_CHECK();
    if (!check(BJ_PART)) {
      // round 0 solved alone, then per launch: apply round r, solve round r + 1
      // (round 0 of the next sweep after the last round)
      int slot = 0;
      hipLaunchKernelGGL(bj_round_kernel, dim3(P), dim3(256), 0, stream, cur, nxt, Vw, lda, m,
                         nbk, -1, nullptr, nullptr, 0, U[0], F[0], P, 0, nullptr);
      FD_LAUNCH_CHECK();
      for (; sweeps < MAX_SWEEPS;) {
        for (int r = 0; r < nbk - 1; ++r) {
          const bool last = r == nbk - 2;
          const int rn = last ? 0 : r + 1;
          hipLaunchKernelGGL(bj_round_kernel, dim3(P + ntile_a + ntile_v), dim3(256), 0, stream,
                             cur, nxt, Vw, lda, m, nbk, r, U[slot], F[slot], rn, U[slot ^ 1],
                             F[slot ^ 1], P, ntile_a, last ? part : nullptr);
          FD_LAUNCH_CHECK();
          std::swap(cur, nxt);
          slot ^= 1;
        }
        ++sweeps;
        if (check(ntile_a)) break;
      }
    }
  }
  // the rotation log / block scratch is free again: it holds the permutation
  check_span_d(log, size_t(m + 1) / 2, "jacobi permutation");
  int* perm = reinterpret_cast<int*>(log.p);
  hipLaunchKernelGGL(jacobi_rank_kernel, dim3(nblk(m, 256)), dim3(256), 0, stream, cur, m, lda,
                     theta, perm);
  FD_LAUNCH_CHECK();
  hipLaunchKernelGGL(jacobi_permute_kernel, dim3(nblk(int64_t(m) * m, 256)), dim3(256), 0, stream,
                     Vw, m, perm, S, lds);
  FD_LAUNCH_CHECK();
  return sweeps;
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

// First-order Loewdin factor of a Gram matrix G (kk x kk, ld ldg) of nearly
// orthonormal columns: L = (3 I - G) / 2, so that (Q L)^T (Q L) = I + O(|G - I|^2).
// Stored in float32 column chunks of width nc (chunk c0 at L + kk c0, element
// (r, c) at r * width + (c - c0)); dev = max |G - I| (one workgroup, fixed order).
__global__ __launch_bounds__(256) void loewdin_kernel(const double* __restrict__ G, int ldg,
                                                      int kk, int nc, float* __restrict__ L,
                                                      double* __restrict__ dev) {
  __shared__ double red[256];
  double mx = 0.0;
  for (int idx = threadIdx.x; idx < kk * kk; idx += blockDim.x) {
    const int r = idx / kk, c = idx % kk;
    const double e = G[int64_t(r) * ldg + c] - (r == c ? 1.0 : 0.0);
    mx = fmax(mx, fabs(e));
    const int c0 = c / nc * nc;
    const int width = min(nc, kk - c0);
    L[int64_t(kk) * c0 + r * width + (c - c0)] = float((r == c ? 1.0 : 0.0) - 0.5 * e);
  }
  red[threadIdx.x] = mx;
  __syncthreads();
  for (int w = blockDim.x / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + w]);
    __syncthreads();
  }
  if (threadIdx.x == 0) *dev = red[0];
}

void loewdin(const double* G, int ldg, int kk, int nc, float* L, double* dev, hipStream_t stream) {
  hipLaunchKernelGGL(loewdin_kernel, dim3(1), dim3(256), 0, stream, G, ldg, kk, nc, L, dev);
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
