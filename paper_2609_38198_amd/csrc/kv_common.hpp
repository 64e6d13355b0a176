// Device-side types and helpers shared by the fused-product translation units.
#pragma once

#include <hip/hip_runtime.h>

#include "fd_internal.hpp"

namespace fd {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __fp16 pkhalf2 __attribute__((ext_vector_type(2)));
typedef unsigned uintx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef _Float16 halfx2 __attribute__((ext_vector_type(2)));

constexpr double LOG2E = 1.4426950408889634073599;
constexpr int CHUNK_TILES = 64;  // column tiles per partial accumulator

// Which of the two layouts of a float32 pack a launch serves (PointPack):
// every launch of such a pair reads the same device word, and the one whose
// layout does not match the exponent budget exits before any work.
struct HxGate {
  const unsigned long long* r2max;
  double bl;    // beta log2(e) of the pack
  int variant;  // 0: no choice, 1: short layout, 2: full-offset layout
};
__device__ __forceinline__ bool hx_gate_closed(const HxGate& g) {
  if (g.variant == 0) return false;
  const double r2 = __longlong_as_double(static_cast<long long>(*g.r2max));
  const bool wide = g.bl * r2 > EXP_BUDGET;
  return wide != (g.variant == 2);
}
inline HxGate gate_of(const PointPack& rows) {
  return HxGate{rows.r2max, rows.beta * LOG2E, rows.variant};
}

// Workgroups of one dispatch are spread over the eight XCDs round-robin by
// id.  Re-number them so that each XCD owns a contiguous block of logical
// work items (same column split, hence a shared working set in its L2).
__device__ __forceinline__ int xcd_remap(int w, int total) {
  if ((total & 7) != 0) return w;
  const int per = total >> 3;
  return (w & 7) * per + (w >> 3);
}

// Split float16 pack of V for one pair of 16-point column tiles: lane (g, p)
// holds rows {4g + r} of the first tile and {16 + 4g + r} of the second
// (r = 0..3) of column 16 cb + p, as hi and lo halves.
struct VSplit {
  halfx8 hi;
  halfx8 lo;
};

// Round two floats toward zero to float16 (hi) and the remainders likewise
// (lo); returns both packed pairs as 32-bit words.
__device__ __forceinline__ void split2(float a, float b, unsigned& hi, unsigned& lo) {
  const pkhalf2 h = __builtin_amdgcn_cvt_pkrtz(a, b);
  const pkhalf2 l = __builtin_amdgcn_cvt_pkrtz(a - float(h[0]), b - float(h[1]));
  hi = __builtin_bit_cast(unsigned, h);
  lo = __builtin_bit_cast(unsigned, l);
}

// The same split with each remainder formed by one mixed-precision FMA,
// k - h = fma(h, m1, k) reading h straight from the packed float16 word (exact
// in float32) and rounded to nearest float16.
// m1 must be -1; it is a run-time value (a kernel argument) so that the
// compiler keeps the FMA form instead of turning it into a subtraction.
__device__ __forceinline__ void split2m(float a, float b, float m1, unsigned& hi, unsigned& lo) {
  const pkhalf2 h = __builtin_amdgcn_cvt_pkrtz(a, b);
  // each remainder rounded straight into its half of the packed word
  // (v_fma_mixlo_f16 / v_fma_mixhi_f16: two instructions instead of two
  // float32 FMAs and a conversion)
  pkhalf2 l;
  l[0] = (_Float16)__builtin_fmaf(float(h[0]), m1, a);
  l[1] = (_Float16)__builtin_fmaf(float(h[1]), m1, b);
  hi = __builtin_bit_cast(unsigned, h);
  lo = __builtin_bit_cast(unsigned, l);
}

inline unsigned blocks_for(int64_t n, int t) { return unsigned(ceil_div(n, t)); }

// ---------------------------------------------------------------- float32 path
// (split float16 exponent contraction; hx_kernels.hip)

// Recipe index and chunk counts of the split-exponent pack for a feature
// dimension D (1 <= D <= 64).
int hx_recipe_for(int64_t D);
int hx_col_chunks(int rid);
int hx_row_chunks(int rid);

void launch_pack_points_hx(const float* X, int64_t n, int64_t D, int64_t ldx, double beta,
                           bool row_side, PointPack& out, const CentreWs* centre,
                           hipStream_t stream);
// Recipe that keeps all three offset pieces for a short recipe that drops the
// third (-1: the recipe keeps them).
int hx_full_offset_recipe(int rid);
void launch_product_hx(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                       const float* vp, const float* colscale, bool diag, const float* sl,
                       float* Y, int64_t ldy, int b, float* part, hipStream_t stream);
void launch_rowsum_hx(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                      const float* wp, bool diag, float* out, float* part, hipStream_t stream);
// Symmetric row sums of one point set (rows.n == cols.n): per-split row partials
// into part ([nsplit][rows.npad]) and column sums added into colfix (64-bit fixed
// point, fix_scale per unit of the shifted kernel 2^15 K; weights in [0, 1]).
// With sq.part set (weighted passes only), the unit-weight sums of the squared
// kernel K^2 (the kernel at twice the bandwidth) go the same way into sq.part
// and sq.colfix, sq.fix_scale per unit of (2^15 K)^2.
void launch_rowsum_sym_hx(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                          const float* wp, float* part, unsigned long long* colfix,
                          double fix_scale, const SymSquares& sq, hipStream_t stream);

// Scheduling pattern for a region holding M matrix instructions and E
// exponentials: each matrix instruction followed by its share of the
// exponentials and V other vector instructions.
template <int M, int E, int V, int m = 0>
__device__ __forceinline__ void sched_interleave() {
  if constexpr (m < M) {
    constexpr int ne = (m + 1) * E / M - m * E / M;
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // matrix
    if constexpr (ne > 0) __builtin_amdgcn_sched_group_barrier(0x400, ne, 0);  // transcendental
    __builtin_amdgcn_sched_group_barrier(0x002, V, 0);  // vector
    sched_interleave<M, E, V, m + 1>();
  }
}

}  // namespace fd
