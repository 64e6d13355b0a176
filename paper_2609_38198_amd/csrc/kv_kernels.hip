// Shared pieces of the fused Gaussian-kernel products: V and weight packs,
// the bfloat16-input kernels, partial-sum reductions, the degree epilogues and
// the host-side planning and dispatch.  The float32-input kernels (split
// float16 exponent contraction) are in hx_kernels.hip.
//
// Operation (FlashDiffusion Sec. 2.1 eq. matmat, Sec. 2.2 eq. tiled_rbf):
//   Y_I = diag(sl_I) * sum_J exp(-beta * ||x_i - x_j||^2) * (sr_J * V_J),
// and the row sums q = K 1, K w of the normalisation (Sec. 2.1).  The N x N
// kernel matrix is never stored.
#include <hip/hip_runtime.h>

#include <cstring>

#include <algorithm>
#include <cmath>

#include "fd_profile.hpp"
#include "kv_common.hpp"

namespace fd {

int padded_dim(int64_t D) {
  static const int dims[] = {4, 8, 12, 16, 24, 32, 48, 64};
  for (int d : dims)
    if (D <= d) return d;
  return 0;
}

// Floats per point of a pack region: large enough for the float32 (split
// float16 chunks of 16 floats) and the bfloat16 pack of any D with this
// padded width; chunk counts grow with D, so the largest D decides.
int pack_floats_per_point(int64_t D) {
  const int dp = padded_dim(D);
  const int dc16 = int(ceil_div(dp, 32)) * 16;
  const int rid = hx_recipe_for(dp);
  const int hx = 16 * std::max(hx_col_chunks(rid), hx_row_chunks(rid));
  return std::max({dp, dc16, hx});
}

PointPack carve_pack(Arena& a, int64_t n, int dp, int64_t pad) {
  PointPack p;
  p.n = n;
  p.npad = round_up(n, pad);
  p.dp = dp;
  p.xp = a.fspan(size_t(p.npad) * pack_floats_per_point(dp));
  p.ap = a.fspan(size_t(p.npad) * 16);  // [tiles][64][4]: 16 floats per point
  p.ar = a.fspan(size_t(p.npad));
  // the full-offset layout of a short recipe: every D of this padded width
  // whose recipe drops the third offset piece takes the same wider recipe
  const int wide = hx_full_offset_recipe(hx_recipe_for(dp == 32 ? 30 : dp == 64 ? 62 : dp));
  if (wide >= 0)
    p.xp2 = a.fspan(size_t(p.npad) * 16 * std::max(hx_col_chunks(wide), hx_row_chunks(wide)));
  return p;
}

// ------------------------------------------------------------------ centring

// Column partial sums of X rows [blk rpb, (blk + 1) rpb) in float64.
__global__ void centre_sum_kernel(const float* __restrict__ X, int64_t n, int D, int64_t ldx,
                                  int64_t rpb, double* __restrict__ part) {
  __shared__ double red[256];
  const int64_t r0 = int64_t(blockIdx.x) * rpb;
  const int64_t r1 = min(n, r0 + rpb);
  for (int f = 0; f < D; ++f) {
    double acc = 0.0;
    for (int64_t i = r0 + threadIdx.x; i < r1; i += blockDim.x) acc += double(X[i * ldx + f]);
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if (int(threadIdx.x) < w) red[threadIdx.x] += red[threadIdx.x + w];
      __syncthreads();
    }
    if (threadIdx.x == 0) part[int64_t(blockIdx.x) * D + f] = red[0];
    __syncthreads();
  }
}

// mu = column means (fixed order over the blocks); clears r2max.
__global__ void centre_mean_kernel(const double* __restrict__ part, int nblk, int D, int64_t n,
                                   double* __restrict__ mu, unsigned long long* r2max) {
  const int f = threadIdx.x;
  if (f == 0) *r2max = 0ull;
  if (f >= D) return;
  double acc = 0.0;
  for (int b = 0; b < nblk; ++b) acc += part[int64_t(b) * D + f];
  mu[f] = acc / double(n);
}

// r2max = max(r2max, max_i ||x_i - mu||^2) over X[0:n] (non-negative float64
// values order like their bit patterns, so an integer atomic max serves).
__global__ void radius_max_kernel(const float* __restrict__ X, int64_t n, int D, int64_t ldx,
                                  const double* __restrict__ mu, unsigned long long* r2max) {
  double best = 0.0;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * blockDim.x) {
    double r = 0.0;
    for (int f = 0; f < D; ++f) {
      const double v = double(X[i * ldx + f]) - mu[f];
      r += v * v;
    }
    best = r > best ? r : best;  // a NaN row is skipped; the non-finite scan reports it
  }
  for (int o = 32; o > 0; o >>= 1) best = fmax(best, __shfl_xor(best, o));
  if ((threadIdx.x & 63) == 0 && best > 0.0)
    atomicMax(r2max, static_cast<unsigned long long>(__double_as_longlong(best)));
}

static int centre_blocks(int64_t n) {
  return int(std::min<int64_t>(256, std::max<int64_t>(1, ceil_div(n, 4096))));
}

CentreWs carve_centre(Arena& a, int64_t n) {
  CentreWs c;
  c.nblk = centre_blocks(n);
  c.part = a.take<double>(size_t(c.nblk) * MAX_D);
  c.mu = a.take<double>(MAX_D);
  c.r2max = a.take<unsigned long long>(1);
  return c;
}

void launch_centre(const void* X, fd_dtype xt, int64_t n, int64_t D, int64_t ldx,
                   const CentreWs& c, hipStream_t stream) {
  if (xt != FD_F32) return;
  FD_REQUIRE(c.part != nullptr && c.mu != nullptr && c.r2max != nullptr && D <= MAX_D &&
                 centre_blocks(n) <= c.nblk,
             FD_ERR_INVALID_ARG, "internal: centring workspace");
  const int nblk = centre_blocks(n);
  const int64_t rpb = ceil_div(n, nblk);
  const float* Xf = static_cast<const float*>(X);
  hipLaunchKernelGGL(centre_sum_kernel, dim3(nblk), dim3(256), 0, stream, Xf, n, int(D), ldx,
                     rpb, c.part);
  FD_LAUNCH_CHECK();
  hipLaunchKernelGGL(centre_mean_kernel, dim3(1), dim3(64), 0, stream, c.part, nblk, int(D), n,
                     c.mu, c.r2max);
  FD_LAUNCH_CHECK();
  launch_radius_more(X, xt, n, D, ldx, c, stream);
}

void launch_radius_more(const void* X2, fd_dtype xt, int64_t n2, int64_t D, int64_t ldx,
                        const CentreWs& c, hipStream_t stream) {
  if (xt != FD_F32) return;
  const unsigned grid = unsigned(std::min<int64_t>(1024, std::max<int64_t>(1, ceil_div(n2, 256))));
  hipLaunchKernelGGL(radius_max_kernel, dim3(grid), dim3(256), 0, stream,
                     static_cast<const float*>(X2), n2, int(D), ldx, c.mu, c.r2max);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------------ exponent range

// f2: the square of the larger coordinate scale (s or 2 beta log2(e) / s)
__global__ void range_check_kernel(const unsigned long long* __restrict__ r2max, double bl,
                                   double f2, int* __restrict__ flag) {
  const double r2 = __longlong_as_double(static_cast<long long>(*r2max));
  if (!(bl * r2 <= HX_EXP_RANGE && f2 * r2 <= HX_PIECE_MAX * HX_PIECE_MAX)) atomicOr(flag, 2);
}

static double coord_scale_sq(double beta) {
  const double s = hx_coord_scale(beta);
  const double f = std::max(s, 2.0 * beta * LOG2E / s);
  return f * f;
}

bool exponent_in_range(fd_dtype xt, double beta, double r2max) {
  return xt != FD_F32 || (beta * LOG2E * r2max <= HX_EXP_RANGE &&
                          coord_scale_sq(beta) * r2max <= HX_PIECE_MAX * HX_PIECE_MAX);
}

double exponent_radius(fd_dtype xt, const CentreWs& c, hipStream_t stream) {
  if (xt != FD_F32) return 0.0;
  unsigned long long bits = 0;
  FD_HIP_CHECK(hipMemcpyAsync(&bits, c.r2max, sizeof(bits), hipMemcpyDeviceToHost, stream));
  FD_HIP_CHECK(hipStreamSynchronize(stream));
  double r2 = 0.0;
  std::memcpy(&r2, &bits, sizeof(r2));
  return r2;
}

void require_exponent_range(fd_dtype xt, const CentreWs& c, double beta, hipStream_t stream) {
  if (xt != FD_F32) return;
  const double r2 = exponent_radius(xt, c, stream);
  if (!exponent_in_range(xt, beta, r2))
    throw Error{FD_ERR_UNSUPPORTED,
                "beta log2(e) max ||x - mean||^2 = " + std::to_string(beta * LOG2E * r2) +
                    " with max ||x - mean|| = " + std::to_string(std::sqrt(r2)) +
                    " is beyond the float32 path's exponent range (offsets up to " +
                    std::to_string(HX_EXP_RANGE) + ", coordinate pieces up to 65504)"};
}

void launch_range_check(fd_dtype xt, const CentreWs& c, double beta, int* flag,
                        hipStream_t stream) {
  if (xt != FD_F32) return;
  FD_REQUIRE(c.r2max != nullptr && flag != nullptr, FD_ERR_INVALID_ARG,
             "internal: range check words");
  hipLaunchKernelGGL(range_check_kernel, dim3(1), dim3(1), 0, stream, c.r2max, beta * LOG2E,
                     coord_scale_sq(beta), flag);
  FD_LAUNCH_CHECK();
}

// ------------------------------------------------------------------ packing

__global__ void pack_w_kernel(const float* __restrict__ w, int64_t n, int64_t ntiles,
                              floatx4* __restrict__ wp) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= ntiles * 64) return;
  const int lane = int(idx & 63);
  const int64_t jb = idx >> 6;
  const int g = lane >> 4;
  floatx4 out;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t j = jb * TILE + 4 * g + r;
    out[r] = (j < n) ? w[j] : 0.f;
  }
  wp[idx] = out;
}

// Weight pack of sr * v for a single right-hand side v (stride ldv): the
// layout of pack_w_kernel.
__global__ void pack_wv_kernel(const float* __restrict__ v, int64_t ldv,
                               const float* __restrict__ sr, int64_t n, int64_t ntiles,
                               floatx4* __restrict__ wp) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= ntiles * 64) return;
  const int lane = int(idx & 63);
  const int64_t jb = idx >> 6;
  const int g = lane >> 4;
  floatx4 out;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t j = jb * TILE + 4 * g + r;
    out[r] = (j < n) ? (sr != nullptr ? sr[j] * v[j * ldv] : v[j * ldv]) : 0.f;
  }
  wp[idx] = out;
}

// Y[i] = sl[i] * t[i] (sl NULL: copy), Y with row stride ldy.
__global__ void scale_rows_kernel(const float* __restrict__ t, const float* __restrict__ sl,
                                  int64_t n, float* __restrict__ Y, int64_t ldy) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) Y[i * ldy] = (sl != nullptr) ? sl[i] * t[i] : t[i];
}

// 2^t clamped to [0, 1]: the exponent of a true kernel value is <= 0 and
// rounding can only push it a few ulps above.  The median-of-three with 0 and 1
// folds into the output clamp bit of v_exp_f32 (one instruction).  Written with
// builtins, not inline asm, so the compiler sees the read of the MFMA result
// and inserts the wait states that hazard requires.
__device__ __forceinline__ float exp2_unit(float t) {
  return __builtin_amdgcn_fmed3f(__builtin_amdgcn_exp2f(t), 0.f, 1.f);
}

// Column-tile operands of one 16-point tile, per lane.
// ------------------------------------------------------------------ split V pack
//
// The K*V contraction runs in float16 with a two-term split of both factors:
//   K' = 2^15 K = Kh + Kl,  V' = 2^e_c sr V = Vh + Vl  (Kh, Kl, Vh, Vl float16),
//   K' V' ~= Kh Vh + Kh Vl + Kl Vh       (the dropped Kl Vl is 2^-22 relative),
// with float32 accumulation; the result is scaled back by 2^(-15 - e_c).  e_c
// puts the largest |V'| of column c just below 2^14; the representation error
// of each split is below 2^-21 relative.  Two consecutive 16-point column tiles
// form the 32-wide contraction; the pack stores, per lane (g, p), the 8 rows
// {4g + r, 16 + 4g + r} of column 16 cb + p as hi and lo halves.

// max |sr_j V[j][c]| per column as float bits (non-negative floats order like
// their bit patterns, so an integer max is exact and order independent)
__global__ void vmax_zero_kernel(unsigned* __restrict__ maxbits) {
  if (threadIdx.x < 64) maxbits[threadIdx.x] = 0u;
}

// Thread (row lane rl, column c): tc = power of two >= b columns side by side
// (consecutive addresses of a row), 256 / tc row lanes; the grid strides over
// the rows, four at a time with their loads issued together; one integer
// atomicMax per column and workgroup.
__global__ __launch_bounds__(256) void vmax_kernel(const float* __restrict__ V, int64_t n, int b,
                                                   int64_t ldv, const float* __restrict__ sr,
                                                   int tc, unsigned* __restrict__ maxbits) {
  __shared__ float red[256];
  const int c = threadIdx.x % tc;
  const int rl = threadIdx.x / tc;
  const int nrl = 256 / tc;
  const int64_t stride = int64_t(gridDim.x) * nrl;
  float m = 0.f;
  if (c < b) {
    for (int64_t i = int64_t(blockIdx.x) * nrl + rl; i < n; i += 4 * stride) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t r = min(i + u * stride, n - 1);
        v[u] = V[r * ldv + c];
        if (sr != nullptr) v[u] *= sr[r];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (i + u * stride < n) m = fmaxf(m, fabsf(v[u]));
    }
  }
  red[threadIdx.x] = m;
  __syncthreads();
  for (int w = 128; w >= tc; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + w]);
    __syncthreads();
  }
  if (threadIdx.x < tc) {
    m = red[threadIdx.x];
    if (c < b && m > 0.f) atomicMax(&maxbits[c], __float_as_uint(m));
  }
}

__device__ __forceinline__ int vscale_exponent(unsigned bits) {
  if (bits == 0u) return 0;
  int e;
  (void)frexpf(__uint_as_float(bits), &e);  // max < 2^e
  return 14 - e;                            // scaled max < 2^14
}

__global__ void pack_v_split_kernel(const float* __restrict__ V, int64_t n, int b, int64_t ldv,
                                    const float* __restrict__ sr, int ncb, int64_t npairs,
                                    const unsigned* __restrict__ maxbits,
                                    VSplit* __restrict__ vp, float* __restrict__ colscale) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= npairs * ncb * 64) return;
  const int lane = int(idx & 63);
  const int cb = int((idx >> 6) % ncb);
  const int64_t jp = idx / (64 * ncb);
  const int g = lane >> 4, p = lane & 15;
  const int c = cb * 16 + p;
  const int ex = (c < b) ? vscale_exponent(maxbits[c]) : 0;
  const float scale = ldexpf(1.f, ex);
  if (jp == 0 && g == 0 && c < b) colscale[c] = ldexpf(1.f, -ex - 15);
  uintx4 hw, lw;
#pragma unroll
  for (int e = 0; e < 8; e += 2) {
    float v[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int ee = e + u;
      const int64_t j = jp * 32 + (ee < 4 ? 4 * g + ee : 16 + 4 * g + (ee - 4));
      float x = 0.f;
      if (j < n && c < b) {
        x = V[j * ldv + c];
        if (sr != nullptr) x *= sr[j];
      }
      v[u] = x * scale;
    }
    unsigned h, l;
    split2(v[0], v[1], h, l);
    hw[e / 2] = h;
    lw[e / 2] = l;
  }
  VSplit out;
  out.hi = __builtin_bit_cast(halfx8, hw);
  out.lo = __builtin_bit_cast(halfx8, lw);
  vp[idx] = out;
}

// Column-pair operands: exponent-contraction inputs of two 16-point tiles and
// the split V pack of the pair.
// ------------------------------------------------------------------ bfloat16 inputs
//
// For X in bfloat16 the exponent contraction runs on v_mfma_f32_16x16x32_bf16:
// products of bfloat16 values are exact in float32, so the tile
//   C[j][i] = -(r_i + r_j) / 2 + x_j . x_i = -||x_i - x_j||^2 / 2
// is computed on raw (unscaled) bfloat16 operands with float32 accumulation,
// and t = 2 beta log2(e) C is applied afterwards on the vector ALUs.  In the
// K*V contraction K' = 2^15 K is rounded once to the nearest float16 (relative
// error <= 2^-12, well inside the bfloat16-input tolerance) and multiplied by
// the split V (hi + lo): the product is then a fixed matrix applied linearly
// to 2^-22, so an eigensolver built on it can converge to its tolerance.
//
// Pack layout (per 16-point tile and 32-feature chunk c): lane (g, p) holds
// the 8 bfloat16 x[16 tile + p][32 c + 8 g + e], e = 0..7, as one uint4; that
// is the A operand of the column tile and the B operand of the row tile.

__global__ void norms_bf16_kernel(const uint16_t* __restrict__ X, int64_t n, int D, int64_t ldx,
                                  float* __restrict__ ap, float* __restrict__ ar, int64_t npad) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= npad) return;
  double r = 0.0;
  if (i < n)
    for (int k = 0; k < D; ++k) {
      const double x = double(__uint_as_float(uint32_t(X[i * ldx + k]) << 16));
      r += x * x;
    }
  // padded points: a huge negative offset makes their kernel values exactly 0
  const float a = (i < n) ? float(-0.5 * r) : -1e30f;
  ar[i] = a;
  if (ap != nullptr) {
    const int64_t tile = i / TILE;
    const int p = int(i % TILE);
    const int g = p >> 2, rr = p & 3;
    float* base = ap + (tile * 64 + 16 * g) * 4 + rr;
    for (int q = 0; q < 16; ++q) base[q * 4] = a;
  }
}

__global__ void pack_bf16_kernel(const uint16_t* __restrict__ X, int64_t n, int D, int64_t ldx,
                                 int dc, int64_t ntiles, uintx4* __restrict__ xp) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= ntiles * dc * 64) return;
  const int lane = int(idx & 63);
  const int c = int((idx >> 6) % dc);
  const int64_t tile = idx / (64 * dc);
  const int g = lane >> 4, p = lane & 15;
  const int64_t i = tile * TILE + p;
  uintx4 out;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t word = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k = 32 * c + 8 * g + 2 * w + h;
      const uint32_t v = (i < n && k < D) ? uint32_t(X[i * ldx + k]) : 0u;
      word |= v << (16 * h);
    }
    out[w] = word;
  }
  xp[idx] = out;
}


template <int DC, bool DIAG>
__device__ __forceinline__ floatx4 half_sqdist(const uintx4* xa, const floatx4& aj,
                                               const uintx4* xb, float ai, int g, int p) {
  floatx4 t;
#pragma unroll
  for (int r = 0; r < 4; ++r) t[r] = ai + aj[r];
#pragma unroll
  for (int c = 0; c < DC; ++c)
    t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, xa[c]),
                                                __builtin_bit_cast(bf16x8, xb[c]), t, 0, 0, 0);
  if (DIAG) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (4 * g + r == p) t[r] = 0.f;
  }
  return t;
}

template <int DC, int NCB>
struct ColPairB {
  uintx4 xa[2][DC];
  floatx4 aj[2];
  VSplit v[NCB];
};

template <int DC, int NCB>
__device__ __forceinline__ void load_pair_b(ColPairB<DC, NCB>& cp, const uintx4* __restrict__ xa,
                                            const floatx4* __restrict__ aj,
                                            const VSplit* __restrict__ vp, int64_t jp, int lane) {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int64_t jb = 2 * jp + t;
#pragma unroll
    for (int c = 0; c < DC; ++c) cp.xa[t][c] = xa[(jb * DC + c) * 64 + lane];
    cp.aj[t] = aj[jb * 64 + lane];
  }
  // unconditional: a branch here would leave the compiler unsure whether the
  // V loads were issued, and its merged load counts would then make every
  // exponent contraction wait for the V loads as well
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) cp.v[cb] = vp[(jp * NCB + cb) * 64 + lane];
}

// Exponents of one pair of column tiles against row tile ib, in accumulator
// layout with the column offsets as the initial accumulator:
//   u_ij = -||x_j||^2 / 2 + x_j . x_i,  K'_ij = 2^(scale2 u_ij + c_i) = 2^15 K_ij,
// with c_i = 15 - scale2 ||x_i||^2 / 2 per row (one FMA per entry).  K' is
// rounded to float16 (nearest, two per instruction) and multiplied into the
// split V on the float16 matrix cores; lane (g, p) holds K'[p][J0 + 4g + r]
// and K'[p][J1 + 4g + r], its A-operand values k = 8g + 4u + r.
template <int DC, bool DIAG>
__device__ __forceinline__ halfx8 bf16_kpair(const uintx4 (&xa)[2][DC], const floatx4 (&aj)[2],
                                             const uintx4 (&xb)[DC], float ci, float scale2,
                                             int64_t jp, int64_t ib, int g, int p) {
  floatx4 t[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    t[u] = aj[u];
#pragma unroll
    for (int cc = 0; cc < DC; ++cc)
      t[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, xa[u][cc]),
                                                     __builtin_bit_cast(bf16x8, xb[cc]), t[u], 0,
                                                     0, 0);
  }
  float e[8];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      e[4 * u + r] = fmaf(t[u][r], scale2, ci);
      // the diagonal of one point set: K'_ii = 2^15 exactly
      if (DIAG && 2 * jp + u == ib && 4 * g + r == p) e[4 * u + r] = 15.f;
    }
  halfx8 k;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const floatx2 kk = floatx2{__builtin_amdgcn_exp2f(e[2 * q]), __builtin_amdgcn_exp2f(e[2 * q + 1])};
    const halfx2 hk = __builtin_convertvector(kk, halfx2);
    k[2 * q] = hk[0];
    k[2 * q + 1] = hk[1];
  }
  return k;
}

template <int NCB>
__device__ __forceinline__ void bf16_kv(const halfx8& k, const VSplit (&v)[NCB],
                                        floatx4 (&acc)[NCB]) {
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(k, v[cb].hi, acc[cb], 0, 0, 0);
    acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(k, v[cb].lo, acc[cb], 0, 0, 0);
  }
}

template <int DC, int NCB, int NIB, bool DIAG>
__device__ __forceinline__ void bf16_pair(const ColPairB<DC, NCB>& c, const uintx4 (&xbr)[NIB][DC],
                                          const float (&ci)[NIB], float scale2,
                                          floatx4 (&acc)[NIB][NCB], int64_t jp, int64_t ib0,
                                          int g, int p) {
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
    const halfx8 k = bf16_kpair<DC, DIAG>(c.xa, c.aj, xbr[ib], ci[ib], scale2, jp, ib0 + ib, g, p);
    bf16_kv<NCB>(k, c.v, acc[ib]);
  }
}

// Waves per SIMD asked of the compiler (at 2 a wave has at most 256
// registers and accumulates in ordinary VGPRs; the widest blocks take 1).
template <int DC, int NCB, int NIB>
constexpr int bf16_waves() {
  constexpr int buffers = NCB >= 3 ? 1 : 2;
  return (NIB * NCB * 4 + NIB * DC * 4 + buffers * (DC * 8 + 8 + NCB * 8) > 200) ? 1 : 2;
}

// One workgroup = 4 waves; wave w owns row tiles [ib0, ib0 + NIB).  Column
// tiles stream in pairs through two operand buffers used in turn (each
// refilled right after its pair is consumed); chunk totals of the two-level
// column sum live in LDS.
template <int DC, int NCB, int NIB>
__global__ __launch_bounds__(WG_THREADS)
__attribute__((amdgpu_waves_per_eu(bf16_waves<DC, NCB, NIB>()))) void product_bf16_kernel(
    const uintx4* __restrict__ xa, const floatx4* __restrict__ aj, const VSplit* __restrict__ vp,
    const uintx4* __restrict__ xb, const float* __restrict__ ar, int64_t nrt, int64_t njp,
    int64_t jp_per_split, int diag, float scale2, const float* __restrict__ colscale,
    const float* __restrict__ sl, float* __restrict__ Y, int64_t ldy, int64_t Nr, int b,
    float* __restrict__ part, int64_t nrpad) {
  __shared__ floatx4 tot[4][NIB][NCB][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t split = wr / nrt;
  const int64_t rt = wr % nrt;
  const int64_t ib0 = (rt * 4 + wave) * NIB;
  const int64_t jp_begin = split * jp_per_split;
  const int64_t jp_end = min(njp, jp_begin + jp_per_split);
  const int g = lane >> 4, p = lane & 15;

  uintx4 xbr[NIB][DC];
  float ci[NIB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
    for (int cc = 0; cc < DC; ++cc) xbr[ib][cc] = xb[((ib0 + ib) * DC + cc) * 64 + lane];
    ci[ib] = fmaf(scale2, ar[(ib0 + ib) * TILE + p], 15.f);
  }
  floatx4 acc[NIB][NCB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      acc[ib][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
      tot[wave][ib][cb][lane] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

  if constexpr (NCB >= 3) {
    // Wide blocks: one buffer each for the exponent operands and for V.  A
    // step first forms K' of all the wave's row tiles (then refills the
    // exponent operands), then multiplies them into V (then refills V); each
    // load has the other phase's work to land, and the registers saved by
    // single buffering keep two waves per SIMD.
    ColPairB<DC, NCB> c;
    load_pair_b(c, xa, aj, vp, jp_begin, lane);
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
      for (int cc = 0; cc < DC; ++cc) asm volatile("" ::"v"(xbr[ib][cc]));
      asm volatile("" ::"v"(ci[ib]));
    }
    int chunk = 0;
    for (int64_t jp = jp_begin; jp < jp_end; ++jp) {
      const int64_t jn = min(jp + 1, jp_end - 1);
      halfx8 k[NIB];
      if (diag && 2 * jp + 1 >= ib0 && 2 * jp < ib0 + NIB) {
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib)
          k[ib] = bf16_kpair<DC, true>(c.xa, c.aj, xbr[ib], ci[ib], scale2, jp, ib0 + ib, g, p);
      } else {
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib)
          k[ib] = bf16_kpair<DC, false>(c.xa, c.aj, xbr[ib], ci[ib], scale2, jp, ib0 + ib, g, p);
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int64_t jb = 2 * jn + t;
#pragma unroll
        for (int cc = 0; cc < DC; ++cc) c.xa[t][cc] = xa[(jb * DC + cc) * 64 + lane];
        c.aj[t] = aj[jb * 64 + lane];
      }
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) bf16_kv<NCB>(k[ib], c.v, acc[ib]);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) c.v[cb] = vp[(jn * NCB + cb) * 64 + lane];
      if (++chunk == CHUNK_TILES / 2) {
        chunk = 0;
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) {
            tot[wave][ib][cb][lane] += acc[ib][cb];
            acc[ib][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
          }
      }
    }
  } else {
  auto step = [&](const ColPairB<DC, NCB>& c, int64_t jp) {
    if (diag && 2 * jp + 1 >= ib0 && 2 * jp < ib0 + NIB)
      bf16_pair<DC, NCB, NIB, true>(c, xbr, ci, scale2, acc, jp, ib0, g, p);
    else
      bf16_pair<DC, NCB, NIB, false>(c, xbr, ci, scale2, acc, jp, ib0, g, p);
  };
  ColPairB<DC, NCB> b0, b1;
  load_pair_b(b0, xa, aj, vp, jp_begin, lane);
  __builtin_amdgcn_sched_barrier(0);  // b0's loads ahead of b1's, as in the loop
  load_pair_b(b1, xa, aj, vp, min(jp_begin + 1, jp_end - 1), lane);
  // consume the row operands before the loop (an empty statement reading
  // them): their loads then complete here, and the loop's waits only ever
  // cover the column buffer a step consumes
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
    for (int cc = 0; cc < DC; ++cc) asm volatile("" ::"v"(xbr[ib][cc]));
    asm volatile("" ::"v"(ci[ib]));
  }
  int chunk = 0;
  for (int64_t jp = jp_begin; jp < jp_end; jp += 2) {
    step(b0, jp);
    // the refills are unconditional (clamped index): every path reaches the
    // loop top with the same loads in flight
    load_pair_b(b0, xa, aj, vp, min(jp + 2, jp_end - 1), lane);
    if (jp + 1 < jp_end) step(b1, jp + 1);
    load_pair_b(b1, xa, aj, vp, min(jp + 3, jp_end - 1), lane);
    chunk += 2;
    if (chunk >= CHUNK_TILES / 2) {
      chunk = 0;
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          tot[wave][ib][cb][lane] += acc[ib][cb];
          acc[ib][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
    }
  }
  }

#pragma unroll
  for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const floatx4 v = tot[wave][ib][cb][lane] + acc[ib][cb];
      const int c = cb * 16 + p;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t i = (ib0 + ib) * TILE + 4 * g + e;
        if (part != nullptr) {
          part[(split * nrpad + i) * (NCB * 16) + c] = v[e];
        } else if (i < Nr && c < b) {
          const float y = v[e] * colscale[c];
          Y[i * ldy + c] = (sl != nullptr) ? y * sl[i] : y;
        }
      }
    }
}


// Row sums for bfloat16 inputs: the same half squared distances, K = 2^t
// clamped to [0, 1], summed (times the weights) on the vector ALUs.  Two waves
// per SIMD (every variant fits 256 registers): the matrix instructions then
// accumulate in VGPRs, with no copies out of accumulation registers (bitwise
// equal results, 13-17% faster bfloat16 degree passes at D = 30 and 64).
template <int DC, int NIB, bool UNIT>
__global__ __launch_bounds__(WG_THREADS) __attribute__((amdgpu_waves_per_eu(2))) void
rowsum_bf16_kernel(
    const uintx4* __restrict__ xa, const floatx4* __restrict__ aj, const floatx4* __restrict__ wp,
    const uintx4* __restrict__ xb, const float* __restrict__ ar, int64_t nrt, int64_t njb,
    int64_t jb_per_split, int diag, float scale2, float* __restrict__ out, int64_t Nr,
    float* __restrict__ part, int64_t nrpad) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wr = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t split = wr / nrt;
  const int64_t rt = wr % nrt;
  const int64_t ib0 = (rt * 4 + wave) * NIB;
  const int64_t jb_begin = split * jb_per_split;
  const int64_t jb_end = min(njb, jb_begin + jb_per_split);
  const int g = lane >> 4, p = lane & 15;

  uintx4 xbr[NIB][DC];
  float ai[NIB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
    for (int c = 0; c < DC; ++c) xbr[ib][c] = xb[((ib0 + ib) * DC + c) * 64 + lane];
    ai[ib] = ar[(ib0 + ib) * TILE + p];
  }
  float acc[NIB], tot[NIB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) acc[ib] = tot[ib] = 0.f;
  int chunk = 0;
  for (int64_t jb = jb_begin; jb < jb_end; ++jb) {
    uintx4 xar[DC];
#pragma unroll
    for (int c = 0; c < DC; ++c) xar[c] = xa[(jb * DC + c) * 64 + lane];
    const floatx4 ajr = aj[jb * 64 + lane];
    floatx4 w4 = floatx4{1.f, 1.f, 1.f, 1.f};
    if (!UNIT) w4 = wp[jb * 64 + lane];
    const bool dtile = diag && jb >= ib0 && jb < ib0 + NIB;
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
      floatx4 t;
      if (dtile && jb == ib0 + ib)
        t = half_sqdist<DC, true>(xar, ajr, xbr[ib], ai[ib], g, p);
      else
        t = half_sqdist<DC, false>(xar, ajr, xbr[ib], ai[ib], g, p);
      float sum = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float k = exp2_unit(t[r] * scale2);
        sum = UNIT ? sum + k : fmaf(k, w4[r], sum);
      }
      acc[ib] += sum;
    }
    if (++chunk == CHUNK_TILES) {
      chunk = 0;
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) {
        tot[ib] += acc[ib];
        acc[ib] = 0.f;
      }
    }
  }
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
    float v = tot[ib] + acc[ib];
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (g == 0) {
      const int64_t i = (ib0 + ib) * TILE + p;
      if (part != nullptr)
        part[split * nrpad + i] = v;
      else if (i < Nr)
        out[i] = v;
    }
  }
}

__global__ void reduce_product_kernel(const float* __restrict__ part, int nsplit, int64_t nrpad,
                                      int width, const float* __restrict__ colscale,
                                      const float* __restrict__ sl, float* __restrict__ Y,
                                      int64_t ldy, int64_t Nr, int b) {
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= Nr * b) return;
  const int64_t i = idx / b;
  const int c = int(idx % b);
  double s = 0.0;
  for (int k = 0; k < nsplit; ++k) s += double(part[(k * nrpad + i) * width + c]);
  if (colscale != nullptr) s *= double(colscale[c]);
  if (sl != nullptr) s *= double(sl[i]);
  Y[i * ldy + c] = float(s);
}

__global__ void reduce_rowsum_kernel(const float* __restrict__ part, int nsplit, int64_t nrpad,
                                     float* __restrict__ out, int64_t Nr) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= Nr) return;
  double s = 0.0;
  for (int k = 0; k < nsplit; ++k) s += double(part[k * nrpad + i]);
  out[i] = float(s);
}

// Symmetric row sums: out_i = sum over splits of the row partials + the
// fixed-point column sums (colfix * 2^-F), in double, fixed order.
__global__ void reduce_rowsum_sym_kernel(const float* __restrict__ part, int nsplit,
                                         int64_t nrpad, const unsigned long long* __restrict__ colfix,
                                         double inv_fix, float* __restrict__ out, int64_t Nr) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= Nr) return;
  double s = 0.0;
  for (int k = 0; k < nsplit; ++k) s += double(part[k * nrpad + i]);
  s += double(static_cast<long long>(colfix[i])) * inv_fix;
  out[i] = float(s);
}

__global__ void zero_u64_kernel(unsigned long long* __restrict__ p, int64_t n) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0ull;
}

// w = q^-alpha
__global__ void pow_neg_kernel(const float* __restrict__ q, int64_t n, double alpha,
                               float* __restrict__ w) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) w[i] = float(pow(double(q[i]), -alpha));
}

// d = w * t, s = w * d^-1/2 (w = q^-alpha recomputed in double from q)
__global__ void degree_finish_kernel(const float* __restrict__ q, const float* __restrict__ t,
                                     int64_t n, double alpha, float* __restrict__ d,
                                     float* __restrict__ s) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const double w = pow(double(q[i]), -alpha);
  const double dd = w * double(t[i]);
  if (d != nullptr) d[i] = float(dd);
  if (s != nullptr) s[i] = float(w / sqrt(dd));
}

// The two normalisation passes on the symmetric path with their epilogues in
// the reductions (same arithmetic, in the same order, as reduce_rowsum_sym +
// pow_neg + pack_w and reduce_rowsum_sym + degree_finish).  One thread per
// padded point; each clears its fixed-point column sum for the next pass.
// Pass 1: q_i, and if wpk is set w_i = q_i^-alpha written to the weight pack
// (pack_w_kernel's layout: w_j in lanes 16 g + p, p = 0..15, component r of
// tile j / 16, j % 16 = 4 g + r; 0 for padding points) for the wnpad points
// of the column pack.
__global__ void degree_reduce_q_kernel(const float* __restrict__ part, int nsplit, int64_t nrpad,
                                       unsigned long long* __restrict__ colfix, double inv_fix,
                                       float* __restrict__ q, int64_t n, int64_t npad,
                                       double alpha, float* __restrict__ wpk, int64_t wnpad) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= npad) return;
  float w = 0.f;
  if (i < n) {
    double sum = 0.0;
    for (int k = 0; k < nsplit; ++k) sum += double(part[k * nrpad + i]);
    sum += double(static_cast<long long>(colfix[i])) * inv_fix;
    const float qi = float(sum);
    q[i] = qi;
    w = float(pow(double(qi), -alpha));
  }
  colfix[i] = 0ull;
  if (wpk != nullptr && i < wnpad) {
    const int64_t jb = i / TILE;
    const int jj = int(i % TILE), g = jj / 4, r = jj % 4;
    float* base = wpk + (jb * 64 + 16 * g) * 4 + r;
#pragma unroll
    for (int p = 0; p < 16; ++p) base[4 * p] = w;
  }
}

// Pass 2: t_i (the weighted row sums), then d_i = w_i t_i and
// s_i = w_i d_i^-1/2 with w_i = q_i^-alpha in double.
__global__ void degree_reduce_ds_kernel(const float* __restrict__ part, int nsplit, int64_t nrpad,
                                        unsigned long long* __restrict__ colfix, double inv_fix,
                                        const float* __restrict__ q, int64_t n, int64_t npad,
                                        double alpha, float* __restrict__ d,
                                        float* __restrict__ s) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= npad) return;
  if (i < n) {
    double sum = 0.0;
    for (int k = 0; k < nsplit; ++k) sum += double(part[k * nrpad + i]);
    sum += double(static_cast<long long>(colfix[i])) * inv_fix;
    const float ti = float(sum);
    const double w = pow(double(q[i]), -alpha);
    const double dd = w * double(ti);
    if (d != nullptr) d[i] = float(dd);
    if (s != nullptr) s[i] = float(w / sqrt(dd));
  }
  colfix[i] = 0ull;
}

// Pass 2 of a dyadic level: degree_reduce_ds_kernel's outputs, and from the
// squared-kernel sums of the same pass the next level's q (K(2 beta) 1, the
// reduction in the same order as degree_reduce_q_kernel's) with its
// w = q^-alpha written to the weight pack as degree_reduce_q_kernel writes it.
__global__ void degree_reduce_dsq_kernel(const float* __restrict__ part, int nsplit,
                                         int64_t nrpad, unsigned long long* __restrict__ colfix,
                                         double inv_fix, const float* __restrict__ q, int64_t n,
                                         int64_t npad, double alpha, float* __restrict__ d,
                                         float* __restrict__ s, const float* __restrict__ part2,
                                         unsigned long long* __restrict__ colfix2,
                                         float* __restrict__ q_next, float* __restrict__ wpk,
                                         int64_t wnpad) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= npad) return;
  float wn = 0.f;
  if (i < n) {
    double sum = 0.0;
    for (int k = 0; k < nsplit; ++k) sum += double(part[k * nrpad + i]);
    sum += double(static_cast<long long>(colfix[i])) * inv_fix;
    const float ti = float(sum);
    const double w = pow(double(q[i]), -alpha);
    const double dd = w * double(ti);
    if (d != nullptr) d[i] = float(dd);
    if (s != nullptr) s[i] = float(w / sqrt(dd));
    double sum2 = 0.0;
    for (int k = 0; k < nsplit; ++k) sum2 += double(part2[k * nrpad + i]);
    sum2 += double(static_cast<long long>(colfix2[i])) * inv_fix;
    const float qn = float(sum2);
    q_next[i] = qn;
    wn = float(pow(double(qn), -alpha));
  }
  colfix[i] = 0ull;
  colfix2[i] = 0ull;
  if (i < wnpad) {
    const int64_t jb = i / TILE;
    const int jj = int(i % TILE), g = jj / 4, r = jj % 4;
    float* base = wpk + (jb * 64 + 16 * g) * 4 + r;
#pragma unroll
    for (int p = 0; p < 16; ++p) base[4 * p] = wn;
  }
}

// sum(q) - n in double, one workgroup, fixed order (deterministic)
__global__ __launch_bounds__(1024) void sum_minus_n_kernel(const float* __restrict__ q, int64_t n,
                                                            double* __restrict__ out) {
  __shared__ double red[1024];
  // four independent partial sums per thread, each over a fixed index set
  double s4[4] = {0.0, 0.0, 0.0, 0.0};
  int64_t i = threadIdx.x;
  for (; i + 3 * 1024 < n; i += 4 * 1024) {
#pragma unroll
    for (int u = 0; u < 4; ++u) s4[u] += double(q[i + u * 1024]);
  }
  for (; i < n; i += 1024) s4[0] += double(q[i]);
  double s = (s4[0] + s4[1]) + (s4[2] + s4[3]);
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (int(threadIdx.x) < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = red[0] - double(n);
}

// ------------------------------------------------------------------ host side

KVPlan plan_tiles(int64_t Nr, int64_t Nc, int dp, int b, int nib) {
  KVPlan p;
  p.dp = dp;
  p.ncb = int(ceil_div(b, 16));
  p.nib = nib;
  p.njb = ceil_div(Nc, TILE);
  const int64_t rows_per_wg = 4 * p.nib * TILE;
  p.nrt = ceil_div(round_up(Nr, ROW_PAD), rows_per_wg);
  // aim for >= 2048 workgroups (eight per CU), keep >= 8 column tiles per split
  const int64_t target = 2048;
  int64_t ns = std::max<int64_t>(1, ceil_div(target, p.nrt));
  ns = std::min<int64_t>(ns, std::max<int64_t>(1, p.njb / 8));
  // at most SPLIT_SPAN_TILES column tiles per workgroup: the workgroups that
  // run together on an XCD start a split together and drift apart as they go;
  // over a shorter span they stay close enough to share column tiles in L2
  ns = std::max<int64_t>(ns, ceil_div(p.njb, SPLIT_SPAN_TILES));
  ns = std::min<int64_t>(ns, 64);
  // splits hold an even number of column tiles (the split product takes them in pairs)
  p.jb_per_split = round_up(ceil_div(p.njb, ns), 2);
  p.nsplit = int(ceil_div(p.njb, p.jb_per_split));
  return p;
}

// Row tiles per wave of the fused product.  Eight for one 16-column block at
// D <= 12 (5% faster than four on the 6-torus, b = 16: two instructions per
// exponent tile leave room for more independent chains); four everywhere else
// (the fastest or tied on every other shape measured: D in {4, 12, 30, 64},
// b in {8 .. 64}; two and eight are 11-17% slower at D = 30, b = 32).
int product_nib(int dp, int ncb) { return (ncb == 1 && dp <= 12) ? 8 : 4; }

KVPlan plan_product(int64_t Nr, int64_t Nc, int dp, int b) {
  return plan_tiles(Nr, Nc, dp, b, product_nib(dp, int(ceil_div(b, 16))));
}

// Row sums: eight row tiles per wave (more independent exponent chains per
// column tile than four; measured faster on every shape).
KVPlan plan_rowsum(int64_t Nr, int64_t Nc, int dp) { return plan_tiles(Nr, Nc, dp, 1, 8); }

// Symmetric row sums (one point set): workgroups of 4 waves x nib row tiles
// own blocks of 64 nib points; a block's column range (its own block and about
// half of the others) is split for >= 2048 workgroups.  nrt holds the number
// of blocks.  From 64 blocks up, splits are whole blocks (at least
// SYM_MIN_SPLITS of them): the workgroups whose windows start at the same
// block then read the same column tiles, and the kernel runs them side by side
// on one XCD so that they share its L2.
KVPlan plan_rowsum_sym(int64_t N, int64_t npad, int dp, int nib) {
  KVPlan p;
  p.dp = dp;
  p.ncb = 1;
  p.nib = nib;
  p.njb = ceil_div(N, TILE);
  const int64_t BT = 4 * nib;
  p.nrt = npad / (BT * TILE);
  const int64_t span_blocks = 1 + (p.nrt - 1) / 2 + (p.nrt % 2 == 0 ? 1 : 0);  // longest range
  const int64_t target = 2048;
  if (p.nrt >= 64) {
    const int64_t ns = std::max<int64_t>(SYM_MIN_SPLITS, ceil_div(target, p.nrt));
    const int64_t jbk = std::max<int64_t>(1, span_blocks / ns);
    p.jb_per_split = jbk * BT;
    p.nsplit = int(ceil_div(span_blocks, jbk));
    return p;
  }
  const int64_t span = BT * span_blocks;
  int64_t ns = std::max<int64_t>(1, ceil_div(target, p.nrt));
  ns = std::min<int64_t>(ns, std::max<int64_t>(1, span / 8));
  ns = std::min<int64_t>(ns, 64);
  p.jb_per_split = round_up(ceil_div(span, ns), 2);
  p.nsplit = int(ceil_div(span, p.jb_per_split));
  return p;
}

size_t sym_part_rows(int64_t npad, int nib) {
  return size_t(plan_rowsum_sym(npad, npad, 4, nib).nsplit) * size_t(npad);
}

static inline size_t lane4_extent(int64_t tiles, int groups) {
  return size_t(tiles) * groups * 64 * 4;
}

static void pack_points_bf16(const uint16_t* X, int64_t n, int64_t D, int64_t ldx, bool row_side,
                             PointPack& out, hipStream_t stream) {
  const int dc = int(ceil_div(D, 32));
  FD_REQUIRE(out.npad % TILE == 0 && out.npad >= n && dc <= 2, FD_ERR_INVALID_ARG,
             "internal: bad bf16 pack geometry");
  const int64_t ntiles = out.npad / TILE;
  check_span(out.xp, size_t(ntiles) * dc * 64 * 4, "bf16 point pack");
  check_span(out.ar, size_t(out.npad), "row offsets");
  if (!row_side) check_span(out.ap, lane4_extent(ntiles, 1), "column offsets");
  hipLaunchKernelGGL(norms_bf16_kernel, dim3(blocks_for(out.npad, 256)), dim3(256), 0, stream, X,
                     n, int(D), ldx, row_side ? nullptr : out.ap.p, out.ar.p, out.npad);
  FD_LAUNCH_CHECK();
  hipLaunchKernelGGL(pack_bf16_kernel, dim3(blocks_for(ntiles * dc * 64, 256)), dim3(256), 0,
                     stream, X, n, int(D), ldx, dc, ntiles, reinterpret_cast<uintx4*>(out.xp.p));
  FD_LAUNCH_CHECK();
  out.bf16 = true;
  out.dc = dc;
}

void launch_pack_points(const void* X, fd_dtype xt, int64_t n, int64_t D, int64_t ldx,
                        double beta, bool row_side, PointPack& out, const CentreWs* centre,
                        hipStream_t stream) {
  out.beta = beta;
  if (xt == FD_BF16) {
    pack_points_bf16(static_cast<const uint16_t*>(X), n, D, ldx, row_side, out, stream);
    out.rid = -1;
    out.rid2 = -1;
    out.variant = 0;
    out.row_side = row_side;
    return;
  }
  out.bf16 = false;
  out.dc = 0;
  FD_REQUIRE(out.dp % 4 == 0 && D <= out.dp, FD_ERR_INVALID_ARG,
             "internal: bad point pack geometry");
  launch_pack_points_hx(static_cast<const float*>(X), n, D, ldx, beta, row_side, out, centre,
                        stream);
}

void launch_pack_w(const float* w, int64_t n, int64_t npad, FSpan wp, hipStream_t stream) {
  FD_REQUIRE(npad % TILE == 0 && npad >= n, FD_ERR_INVALID_ARG, "internal: bad w pack geometry");
  const int64_t ntiles = npad / TILE;
  check_span(wp, lane4_extent(ntiles, 1), "weight pack");
  hipLaunchKernelGGL(pack_w_kernel, dim3(blocks_for(ntiles * 64, 256)), dim3(256), 0, stream, w,
                     n, ntiles, reinterpret_cast<floatx4*>(wp.p));
  FD_LAUNCH_CHECK();
}

void launch_pack_wv(const float* v, int64_t ldv, const float* sr, int64_t n, int64_t npad,
                    FSpan wp, hipStream_t stream) {
  FD_REQUIRE(npad % TILE == 0 && npad >= n, FD_ERR_INVALID_ARG, "internal: bad w pack geometry");
  const int64_t ntiles = npad / TILE;
  check_span(wp, lane4_extent(ntiles, 1), "weight pack");
  hipLaunchKernelGGL(pack_wv_kernel, dim3(blocks_for(ntiles * 64, 256)), dim3(256), 0, stream, v,
                     ldv, sr, n, ntiles, reinterpret_cast<floatx4*>(wp.p));
  FD_LAUNCH_CHECK();
}

void launch_scale_rows(const float* t, const float* sl, int64_t n, float* Y, int64_t ldy,
                       hipStream_t stream) {
  hipLaunchKernelGGL(scale_rows_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, t, sl, n,
                     Y, ldy);
  FD_LAUNCH_CHECK();
}

// Geometry shared by the product and row-sum launches.
static void check_tiles(const KVPlan& p, const PointPack& rows, const PointPack& cols) {
  const int64_t row_tiles = p.nrt * 4 * p.nib;  // 16-row tiles the grid reads
  FD_REQUIRE(rows.dp == p.dp && cols.dp == p.dp, FD_ERR_INVALID_ARG, "internal: pack width");
  FD_REQUIRE(row_tiles * TILE == rows.npad, FD_ERR_INVALID_ARG,
             "internal: row pack not padded to the workgroup tile");
  FD_REQUIRE(p.njb * TILE <= cols.npad && cols.n <= p.njb * TILE, FD_ERR_INVALID_ARG,
             "internal: column pack does not match the plan");
  FD_REQUIRE(p.nsplit >= 1 && (p.nsplit - 1) * p.jb_per_split < p.njb &&
                 p.nsplit * p.jb_per_split >= p.njb,
             FD_ERR_INVALID_ARG, "internal: bad column split");
  if (rows.bf16) {
    check_span(rows.xp, size_t(row_tiles) * rows.dc * 64 * 4, "bf16 row pack");
    check_span(cols.xp, size_t(round_up(p.njb, 2)) * cols.dc * 64 * 4, "bf16 column pack");
    check_span(rows.ar, size_t(rows.npad), "row offsets");
    check_span(cols.ap, lane4_extent(round_up(p.njb, 2), 1), "column offsets");
  }
}

void launch_pack_v_split(const float* V, int64_t n, int64_t b, int64_t ldv, const float* sr,
                         int ncb, int64_t npad, FSpan vp, FSpan vscale, hipStream_t stream) {
  FD_REQUIRE(npad % (2 * TILE) == 0 && npad >= n && b <= ncb * 16 && b <= 64, FD_ERR_INVALID_ARG,
             "internal: bad split V pack geometry");
  const int64_t npairs = npad / (2 * TILE);
  // one VSplit (32 bytes = 8 floats) per lane per pair per column block
  check_span(vp, size_t(npairs) * ncb * 64 * 8, "split V pack");
  check_span(vscale, 128, "column scales");
  unsigned* maxbits = reinterpret_cast<unsigned*>(vscale.p);
  float* colscale = vscale.p + 64;
  hipLaunchKernelGGL(vmax_zero_kernel, dim3(1), dim3(64), 0, stream, maxbits);
  FD_LAUNCH_CHECK();
  int tc = 1;
  while (tc < b) tc *= 2;
  const int64_t nrl = 256 / tc;
  const unsigned vgrid = unsigned(std::min<int64_t>(256, std::max<int64_t>(1, (n + 4 * nrl - 1) / (4 * nrl))));
  hipLaunchKernelGGL(vmax_kernel, dim3(vgrid), dim3(256), 0, stream, V, n, int(b), ldv, sr, tc,
                     maxbits);
  FD_LAUNCH_CHECK();
  const int64_t total = npairs * ncb * 64;
  hipLaunchKernelGGL(pack_v_split_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, stream, V,
                     n, int(b), ldv, sr, ncb, npairs, maxbits, reinterpret_cast<VSplit*>(vp.p),
                     colscale);
  FD_LAUNCH_CHECK();
}

void launch_pack_v_for(const PointPack& /*rows*/, const float* V, int64_t n, int64_t b,
                       int64_t ldv, const float* sr, int ncb, int64_t npad, FSpan vp,
                       FSpan vscale, hipStream_t stream) {
  // both product kinds take the split V (hi + lo float16 halves)
  launch_pack_v_split(V, n, b, ldv, sr, ncb, npad, vp, vscale, stream);
}

template <int DC, int NCB, int NIB>
static void product_bf16_nib(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                             const float* vp, const float* colscale, bool diag, const float* sl,
                             float* Y, int64_t ldy, int b, float* part, hipStream_t stream) {
  const unsigned grid = unsigned(p.nrt * p.nsplit);
  const float scale2 = float(2.0 * rows.beta * LOG2E);
  ProfScope prof(FD_KERNEL_PRODUCT, stream);
  hipLaunchKernelGGL((product_bf16_kernel<DC, NCB, NIB>), dim3(grid), dim3(WG_THREADS), 0, stream,
                     reinterpret_cast<const uintx4*>(cols.xp.p),
                     reinterpret_cast<const floatx4*>(cols.ap.p),
                     reinterpret_cast<const VSplit*>(vp),
                     reinterpret_cast<const uintx4*>(rows.xp.p), rows.ar.p, p.nrt,
                     ceil_div(p.njb, 2), p.jb_per_split / 2, int(diag), scale2, colscale, sl, Y,
                     ldy, rows.n, b, part, rows.npad);
  FD_LAUNCH_CHECK();
}

template <int DC, int NCB>
static void product_bf16_launch(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                                const float* vp, const float* cs, bool diag, const float* sl,
                                float* Y, int64_t ldy, int b, float* part, hipStream_t stream) {
  // eight row tiles per wave only for the shapes product_nib gives them to
  if constexpr (DC == 1 && NCB == 1) {
    if (p.nib == 8)
      return product_bf16_nib<DC, NCB, 8>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part,
                                          stream);
  }
  FD_REQUIRE(p.nib == 2 || p.nib == 4, FD_ERR_INVALID_ARG, "internal: bf16 rows per wave");
  if (p.nib == 2)
    product_bf16_nib<DC, NCB, 2>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
  else
    product_bf16_nib<DC, NCB, 4>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
}

template <int DC>
static void product_bf16_ncb(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                             const float* vp, const float* cs, bool diag, const float* sl,
                             float* Y, int64_t ldy, int b, float* part, hipStream_t stream) {
  switch (p.ncb) {
    case 1: return product_bf16_launch<DC, 1>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
    case 2: return product_bf16_launch<DC, 2>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
    case 3: return product_bf16_launch<DC, 3>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
    case 4: return product_bf16_launch<DC, 4>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
  }
  throw Error{FD_ERR_UNSUPPORTED, "block width above 64"};
}

void launch_product(const KVPlan& p, const PointPack& rows, const PointPack& cols, FSpan vp,
                    FSpan vscale, bool diag, const float* sl, float* Y, int64_t ldy, int b,
                    FSpan part, hipStream_t stream) {
  check_tiles(p, rows, cols);
  FD_REQUIRE(b >= 1 && b <= p.ncb * 16 && (p.nib == 2 || p.nib == 4 || p.nib == 8),
             FD_ERR_INVALID_ARG, "internal: block width does not match the plan");
  FD_REQUIRE(p.jb_per_split % 2 == 0 && round_up(p.njb, 2) * TILE <= cols.npad,
             FD_ERR_INVALID_ARG, "internal: column pairs do not fit the pack");
  check_span(vscale, 128, "column scales");
  const float* cs = vscale.p + 64;
  float* pp = nullptr;
  if (p.nsplit > 1) {
    check_span(part, size_t(p.nsplit) * rows.npad * p.ncb * 16, "partial products");
    pp = part.p;
  }
  if (rows.bf16 || cols.bf16) {
    FD_REQUIRE(rows.bf16 && cols.bf16 && rows.dc == cols.dc, FD_ERR_INVALID_ARG,
               "internal: mixed pack kinds");
    check_span(vp, size_t(ceil_div(p.njb, 2)) * p.ncb * 64 * 8, "split V pack");
    if (rows.dc == 1)
      product_bf16_ncb<1>(p, rows, cols, vp.p, cs, diag, sl, Y, ldy, b, pp, stream);
    else
      product_bf16_ncb<2>(p, rows, cols, vp.p, cs, diag, sl, Y, ldy, b, pp, stream);
  } else {
    check_span(vp, size_t(ceil_div(p.njb, 2)) * p.ncb * 64 * 8, "split V pack");
    launch_product_hx(p, rows, cols, vp.p, cs, diag, sl, Y, ldy, b, pp, stream);
  }
  if (p.nsplit > 1) {
    const int64_t total = rows.n * b;
    hipLaunchKernelGGL(reduce_product_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, stream,
                       pp, p.nsplit, rows.npad, p.ncb * 16, cs, sl, Y, ldy, rows.n, b);
    FD_LAUNCH_CHECK();
  }
}

template <int DC, int NIB, bool UNIT>
static void rowsum_bf16_nib(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                            const float* wp, bool diag, float* out, float* part,
                            hipStream_t stream) {
  const unsigned grid = unsigned(p.nrt * p.nsplit);
  const float scale2 = float(2.0 * rows.beta * LOG2E);
  ProfScope prof(FD_KERNEL_ROWSUM, stream);
  hipLaunchKernelGGL((rowsum_bf16_kernel<DC, NIB, UNIT>), dim3(grid), dim3(WG_THREADS), 0, stream,
                     reinterpret_cast<const uintx4*>(cols.xp.p),
                     reinterpret_cast<const floatx4*>(cols.ap.p),
                     reinterpret_cast<const floatx4*>(wp),
                     reinterpret_cast<const uintx4*>(rows.xp.p), rows.ar.p, p.nrt, p.njb,
                     p.jb_per_split, int(diag), scale2, out, rows.n, part, rows.npad);
  FD_LAUNCH_CHECK();
}

template <int DC, bool UNIT>
static void rowsum_bf16_launch(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                               const float* wp, bool diag, float* out, float* part,
                               hipStream_t stream) {
  if (p.nib == 8)
    rowsum_bf16_nib<DC, 8, UNIT>(p, rows, cols, wp, diag, out, part, stream);
  else
    rowsum_bf16_nib<DC, 4, UNIT>(p, rows, cols, wp, diag, out, part, stream);
}


bool rowsum_sym_applies(const PointPack& rows, const PointPack& cols, bool diag,
                        const unsigned long long* colfix) {
  return colfix != nullptr && diag && !rows.bf16 && !cols.bf16 && rows.n == cols.n;
}

SymPass launch_rowsum_sym_pass(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                               FSpan wp, FSpan part, unsigned long long* colfix, bool zero_colfix,
                               hipStream_t stream, FSpan sq_part, unsigned long long* sq_colfix) {
  check_tiles(p, rows, cols);
  FD_REQUIRE(rowsum_sym_applies(rows, cols, true, colfix), FD_ERR_INVALID_ARG,
             "internal: symmetric row sums need one float32 point set");
  const KVPlan sp = plan_rowsum_sym(rows.n, rows.npad, p.dp, SYM_NIB);
  if (wp.p != nullptr) check_span(wp, lane4_extent(sp.njb, 1), "weight pack");
  check_span(part, size_t(sp.nsplit) * rows.npad, "partial row sums");
  // fixed point with F fractional bits: the total of weights in [0, 1] over
  // npad columns stays below 2^62 / 4
  const int F = 62 - int(std::ceil(std::log2(double(rows.npad)))) - 2;
  if (zero_colfix) {
    hipLaunchKernelGGL(zero_u64_kernel, dim3(blocks_for(rows.npad, 256)), dim3(256), 0, stream,
                       colfix, rows.npad);
    FD_LAUNCH_CHECK();
  }
  SymSquares sq;
  if (sq_part.p != nullptr) {
    FD_REQUIRE(wp.p != nullptr && sq_colfix != nullptr, FD_ERR_INVALID_ARG,
               "internal: squared sums ride on a weighted pass");
    check_span(sq_part, size_t(sp.nsplit) * rows.npad, "partial squared row sums");
    // (2^15 K)^2 per unit: K^2 <= 1 keeps the same headroom as the weights
    sq = SymSquares{sq_part.p, sq_colfix, std::ldexp(1.0, F - 30)};
  }
  launch_rowsum_sym_hx(sp, rows, cols, wp.p, part.p, colfix, std::ldexp(1.0, F - 15), sq, stream);
  return SymPass{int(sp.nsplit), std::ldexp(1.0, -F)};
}

void launch_degree_reduce_q(const SymPass& sp, const PointPack& rows, const PointPack& cols,
                            FSpan part, unsigned long long* colfix, float* q, double alpha,
                            FSpan wp, hipStream_t stream) {
  FD_REQUIRE(cols.npad % TILE == 0 && cols.npad <= rows.npad && cols.n == rows.n,
             FD_ERR_INVALID_ARG, "internal: bad weight pack geometry");
  if (wp.p != nullptr) check_span(wp, lane4_extent(cols.npad / TILE, 1), "weight pack");
  hipLaunchKernelGGL(degree_reduce_q_kernel, dim3(blocks_for(rows.npad, 256)), dim3(256), 0,
                     stream, part.p, sp.nsplit, rows.npad, colfix, sp.inv_fix, q, rows.n,
                     rows.npad, alpha, wp.p, cols.npad);
  FD_LAUNCH_CHECK();
}

void launch_degree_reduce_ds(const SymPass& sp, const PointPack& rows, FSpan part,
                             unsigned long long* colfix, const float* q, double alpha, float* d,
                             float* s, hipStream_t stream) {
  hipLaunchKernelGGL(degree_reduce_ds_kernel, dim3(blocks_for(rows.npad, 256)), dim3(256), 0,
                     stream, part.p, sp.nsplit, rows.npad, colfix, sp.inv_fix, q, rows.n,
                     rows.npad, alpha, d, s);
  FD_LAUNCH_CHECK();
}

void launch_degree_reduce_dsq(const SymPass& sp, const PointPack& rows, const PointPack& cols,
                              FSpan part, unsigned long long* colfix, const float* q,
                              double alpha, float* d, float* s, FSpan sq_part,
                              unsigned long long* sq_colfix, float* q_next, FSpan wp,
                              hipStream_t stream) {
  FD_REQUIRE(cols.npad % TILE == 0 && cols.npad <= rows.npad && cols.n == rows.n,
             FD_ERR_INVALID_ARG, "internal: bad weight pack geometry");
  check_span(wp, lane4_extent(cols.npad / TILE, 1), "weight pack");
  check_span(sq_part, size_t(sp.nsplit) * rows.npad, "partial squared row sums");
  FD_REQUIRE(q_next != nullptr && sq_colfix != nullptr, FD_ERR_INVALID_ARG,
             "internal: dyadic reduction outputs");
  hipLaunchKernelGGL(degree_reduce_dsq_kernel, dim3(blocks_for(rows.npad, 256)), dim3(256), 0,
                     stream, part.p, sp.nsplit, rows.npad, colfix, sp.inv_fix, q, rows.n,
                     rows.npad, alpha, d, s, sq_part.p, sq_colfix, q_next, wp.p, cols.npad);
  FD_LAUNCH_CHECK();
}

void launch_zero_u64(unsigned long long* p, int64_t n, hipStream_t stream) {
  hipLaunchKernelGGL(zero_u64_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, p, n);
  FD_LAUNCH_CHECK();
}

void launch_rowsum(const KVPlan& p, const PointPack& rows, const PointPack& cols, FSpan wp,
                   bool diag, float* out, FSpan part, hipStream_t stream,
                   unsigned long long* colfix) {
  check_tiles(p, rows, cols);
  if (rowsum_sym_applies(rows, cols, diag, colfix)) {
    // one point set: each off-diagonal tile serves its rows and its columns
    const SymPass sp = launch_rowsum_sym_pass(p, rows, cols, wp, part, colfix, true, stream);
    hipLaunchKernelGGL(reduce_rowsum_sym_kernel, dim3(blocks_for(rows.n, 256)), dim3(256), 0,
                       stream, part.p, sp.nsplit, rows.npad, colfix, sp.inv_fix, out, rows.n);
    FD_LAUNCH_CHECK();
    return;
  }
  FD_REQUIRE(p.nib == 4 || p.nib == 8, FD_ERR_INVALID_ARG, "internal: row-sum plan");
  if (wp.p != nullptr) check_span(wp, lane4_extent(p.njb, 1), "weight pack");
  float* pp = nullptr;
  if (p.nsplit > 1) {
    check_span(part, size_t(p.nsplit) * rows.npad, "partial row sums");
    pp = part.p;
  }
  if (rows.bf16 || cols.bf16) {
    FD_REQUIRE(rows.bf16 && cols.bf16 && rows.dc == cols.dc, FD_ERR_INVALID_ARG,
               "internal: mixed pack kinds");
    const bool unit = wp.p == nullptr;
    if (rows.dc == 1)
      unit ? rowsum_bf16_launch<1, true>(p, rows, cols, wp.p, diag, out, pp, stream)
           : rowsum_bf16_launch<1, false>(p, rows, cols, wp.p, diag, out, pp, stream);
    else
      unit ? rowsum_bf16_launch<2, true>(p, rows, cols, wp.p, diag, out, pp, stream)
           : rowsum_bf16_launch<2, false>(p, rows, cols, wp.p, diag, out, pp, stream);
  } else {
    launch_rowsum_hx(p, rows, cols, wp.p, diag, out, pp, stream);
  }
  if (p.nsplit > 1) {
    hipLaunchKernelGGL(reduce_rowsum_kernel, dim3(blocks_for(rows.n, 256)), dim3(256), 0, stream,
                       pp, p.nsplit, rows.npad, out, rows.n);
    FD_LAUNCH_CHECK();
  }
}

void launch_pow_neg(const float* q, int64_t n, double alpha, float* w, hipStream_t stream) {
  hipLaunchKernelGGL(pow_neg_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, q, n, alpha,
                     w);
  FD_LAUNCH_CHECK();
}

void launch_degree_finish(const float* q, const float* t, int64_t n, double alpha, float* d,
                          float* s, hipStream_t stream) {
  hipLaunchKernelGGL(degree_finish_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, q, t,
                     n, alpha, d, s);
  FD_LAUNCH_CHECK();
}

void launch_sum_minus_n(const float* q, int64_t n, double* out, hipStream_t stream) {
  hipLaunchKernelGGL(sum_minus_n_kernel, dim3(1), dim3(1024), 0, stream, q, n, out);
  FD_LAUNCH_CHECK();
}

}  // namespace fd
