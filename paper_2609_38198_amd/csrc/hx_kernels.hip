// Fused Gaussian-kernel products for float32 inputs on gfx950 matrix cores.
//
// Operation (FlashDiffusion Sec. 2.1 eq. matmat, Sec. 2.2 eq. tiled_rbf):
//   Y_I = diag(sl_I) * sum_J K_IJ * (sr_J * V_J),  K_ij = exp(-beta ||x_i - x_j||^2),
// with the exponent in the Gram form (eq. rbf_gram), in log2 units:
//   t_ij = a_i + a_j + sum_k x_jk b_ik,  a = -beta log2(e) ||x||^2,  b = 2 beta log2(e) x,
// and K_ij = 2^t_ij.  The N x N kernel matrix is never stored: each 16 x 16
// tile lives in four registers of one wave between two matrix-core steps.
//
// Exponent contraction in float16 pieces.  Every float32 coordinate x' (and
// every b', computed in float64) is written as three float16 pieces
// v = v1 + v2 + v3 (each the round-to-nearest float16 of the remainder), which
// represents a float32 value exactly (33 >= 24 significant bits) unless a piece
// underflows.  Products of float16 values are exact in float32.  For D <= 4
// the contraction keeps the six products whose pieces sum to at most four
// (x1 b1, x2 b1, x1 b2, x3 b1, x1 b3, x2 b2; the dropped ones are below 2^-30
// of the term), so the exponent carries only the float32 accumulation rounding.
// For larger D it keeps x1 b1, x2 b1 and x1 b2 (and x3 b1 where it fits for
// free): the dropped products are at most 3 * 2^-22 of |x_jk b_ik| each, the
// order of the float32 rounding of the Gram-form sum itself, for half the
// matrix instructions.  The offsets a_i and a_j enter the same contraction as
// float16 pieces (three, or two where the third does not fit), multiplied by
// slots holding 1, and sit in the first instruction next to x1 b1 so the large
// Gram terms cancel early.  x' = s x and b' = b / s with s = 2^e,
// e ~ log2(2 beta log2 e) / 2, keep both operands near the same magnitude; s
// cancels exactly in x' . b'.
//
// Why float16: on gfx950 a v_mfma_f32_16x16x32_f16 (32 slots) issues every 16
// cycles per SIMD, a v_mfma_f32_16x16x4_f32 (4 slots) every 32.  Measured on
// the device, a matrix instruction holds off ordinary vector instructions of
// the SIMD for most of its duration (the exponentials overlap it only in
// part), so a tile costs about the sum of its instruction times and the
// cheaper float16 contraction (2 instructions for D <= 13 instead of 4 float32
// ones at twice the cost each) shortens it directly.
//
// Pack layout (both sides): per 16-point tile and 32-slot chunk c, lane (g, p)
// holds slots 8g .. 8g+7 of point 16 tile + p as eight float16 values (one
// uint4): the A operand of v_mfma_f32_16x16x32_f16 for a column tile, the B
// operand for a row tile.  A recipe (table below, per range of D) says which
// piece or constant each slot holds and which (column chunk, row chunk) pairs
// the contraction multiplies.  The accumulator then holds T^T[4g + r][p], the
// layout the K*V step consumes without data movement (see product_hx_kernel).
//
// K*V contraction: float16 two-term split of both factors,
//   K' = 2^15 K = Kh + Kl,  V' = 2^e_c sr V = Vh + Vl,  K'V' ~= Kh Vh + Kh Vl + Kl Vh,
// on v_mfma_f32_16x16x32_f16 with float32 accumulation; the result is scaled
// back by 2^(-15 - e_c).  The shift 15 is folded into the row-side offset
// pieces (a_i + 15), so both the product and the row sums work with
// K' = 2^15 K (the row sums scale back by 2^-15, exactly).  Sums over columns
// are two-level (a fresh accumulator per 64 column tiles added into a running
// total).  When rows and columns are the same point set the diagonal exponent
// is set to its exact value (K'_ii = 2^15).
//
// Accuracy condition (either contraction form): the Gram form cancels terms of
// size beta ||x||^2; inputs should be centred so that this stays moderate
// (float32 resolves t to about 2^-24 beta log2(e) max ||x||^2, the short split
// to a small multiple of 2^-22 of it).  Pieces are
// saturated to the float16 range, so even beyond that every value is finite.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "fd_profile.hpp"
#include "kv_common.hpp"

namespace fd {

namespace {

// ------------------------------------------------------------------ recipes

enum : int8_t { SEG_END = 0, SEG_X = 1, SEG_ONES = 2, SEG_A = 3 };

// A run of slots: SEG_X holds piece `piece` of features foff .. foff+cap-1
// (zero past D); SEG_ONES holds cap 1s; SEG_A holds pieces piece .. piece+cap-1
// of the offset a.
struct HxSeg {
  int8_t kind, piece, slot, cap, foff;
};
constexpr int HX_SEGS = 8, HX_CHUNKS = 5, HX_MFMAS = 7, HX_RECIPES = 7;
struct HxChunk {
  HxSeg s[HX_SEGS];
};
struct HxSide {
  HxChunk ch[HX_CHUNKS];
};
// nc / nb: chunks per column / row point; instruction m multiplies column
// chunk sa[m] by row chunk sb[m].  order: the recipe holds every piece product
// x_p b_q with p + q <= order (4: the exact split, 3: the short split).
struct HxRecipe {
  int8_t maxd, nc, nb, nm, order;
  int8_t sa[HX_MFMAS], sb[HX_MFMAS];
  HxSide col, row;
};

constexpr HxSeg X(int piece, int slot, int cap, int foff = 0) {
  return HxSeg{SEG_X, int8_t(piece), int8_t(slot), int8_t(cap), int8_t(foff)};
}
constexpr HxSeg ONES(int slot, int cap = 3) {
  return HxSeg{SEG_ONES, 0, int8_t(slot), int8_t(cap), 0};
}
constexpr HxSeg AOF(int slot) { return HxSeg{SEG_A, 1, int8_t(slot), 3, 0}; }
// single piece k of the offset
constexpr HxSeg APC(int slot, int k) { return HxSeg{SEG_A, int8_t(k), int8_t(slot), 1, 0}; }

// Column side: x pieces, a_j against row-side 1s; row side: b pieces, a_i
// against column-side 1s.  Slot by slot the column and row chunks of each
// instruction pair as (x_p, b_q), (1, a_i) or (a_j, 1); every other slot
// pairing has a zero on one side.
//
// D <= 4 fits the exact split in one instruction.  Above that the recipes
// keep the products of order p + q <= 3 (x1 b1, x2 b1, x1 b2) and the offset
// pieces 1 and 2, plus what fits in the same instructions for free (x3 b1 and
// the third offset pieces for some D).  The dropped terms are at most
// 3 * 2^-22 |x_jk b_ik| per feature and 2^-22 |a| per offset, the order of the
// float32 rounding of the Gram-form sum itself, and the contraction needs
// about half the instructions of the exact split.
constexpr HxRecipe HX_TABLE[HX_RECIPES] = {
    // D <= 4: one instruction, exact split
    {4, 1, 1, 1, 4, {0}, {0},
     {{{{X(1, 0, 4), X(2, 4, 4), X(1, 8, 4), X(3, 12, 4), X(1, 16, 4), X(2, 20, 4), ONES(24),
         AOF(27)}}}},
     {{{{X(1, 0, 4), X(1, 4, 4), X(2, 8, 4), X(1, 12, 4), X(3, 16, 4), X(2, 20, 4), AOF(24),
         ONES(27)}}}}},
    // D <= 8: x1b1 + x2b1 + x1b2 + a_i + a_j in one instruction
    {8, 1, 1, 1, 3, {0}, {0},
     {{{{X(1, 0, 8), X(2, 8, 8), X(1, 16, 8), ONES(24), AOF(27)}}}},
     {{{{X(1, 0, 8), X(1, 8, 8), X(2, 16, 8), AOF(24), ONES(27)}}}}},
    // D <= 13: x1b1 + a_i + x2b1 + a_j, then x1b2 + x3b1 (column chunk 0
    // pairs with row chunk 0, column chunk 1 with row chunk 1)
    {13, 2, 2, 2, 3, {0, 1}, {0, 1},
     {{{{X(1, 0, 13), ONES(13), X(2, 16, 13), AOF(29)}},
       {{X(1, 0, 13), X(3, 16, 13)}}}},
     {{{{X(1, 0, 13), AOF(13), X(1, 16, 13), ONES(29)}},
       {{X(2, 0, 13), X(1, 16, 13)}}}}},
    // D <= 30: one piece per chunk; the offsets use the two spare slots of
    // each chunk.  Slot 30: 1 on x1 against a_i1, a_i2 on b1, b2; slot 31:
    // a_j1, a_j2 on x1, x2 against 1 on b1.  The three instructions meet each
    // of these offset pieces exactly once.
    {30, 2, 2, 3, 3, {0, 1, 0}, {0, 0, 1},
     {{{{X(1, 0, 30), ONES(30, 1), APC(31, 1)}}, {{X(2, 0, 30), APC(31, 2)}}}},
     {{{{X(1, 0, 30), APC(30, 1), ONES(31, 1)}}, {{X(2, 0, 30), APC(30, 2)}}}}},
    // D <= 32: offsets in a chunk of their own
    {32, 3, 3, 4, 3, {0, 2, 1, 0}, {0, 2, 0, 1},
     {{{{X(1, 0, 32)}}, {{X(2, 0, 32)}}, {{ONES(0), AOF(3)}}}},
     {{{{X(1, 0, 32)}}, {{X(2, 0, 32)}}, {{AOF(0), ONES(3)}}}}},
    // D <= 62: two chunks per piece; the offsets take the spare slots of the
    // second chunks, laid out as for D <= 30
    {62, 4, 4, 6, 3, {0, 1, 2, 3, 0, 1}, {0, 1, 0, 1, 2, 3},
     {{{{X(1, 0, 32)}}, {{X(1, 0, 30, 32), ONES(30, 1), APC(31, 1)}}, {{X(2, 0, 32)}},
       {{X(2, 0, 30, 32), APC(31, 2)}}}},
     {{{{X(1, 0, 32)}}, {{X(1, 0, 30, 32), APC(30, 1), ONES(31, 1)}}, {{X(2, 0, 32)}},
       {{X(2, 0, 30, 32), APC(30, 2)}}}}},
    // D <= 64: two chunks per piece, offsets in a chunk of their own
    {64, 5, 5, 7, 3, {0, 1, 4, 2, 3, 0, 1}, {0, 1, 4, 0, 1, 2, 3},
     {{{{X(1, 0, 32)}}, {{X(1, 0, 32, 32)}}, {{X(2, 0, 32)}}, {{X(2, 0, 32, 32)}},
       {{ONES(0), AOF(3)}}}},
     {{{{X(1, 0, 32)}}, {{X(1, 0, 32, 32)}}, {{X(2, 0, 32)}}, {{X(2, 0, 32, 32)}},
       {{AOF(0), ONES(3)}}}}},
};

// ------------------------------------------------------------------ recipe check
//
// Compile-time proof that every recipe contracts
//   sum_f sum_{p + q <= order} x_p[f] b_q[f] + (a_i1 + a_i2 [+ a_i3]) + (a_j1 + a_j2 [+ a_j3])
// plus possibly some of the higher products (p + q = 4) and third offset
// pieces, for all features f < maxd: over the instructions' (column chunk,
// row chunk) pairs, slot by slot, each wanted product appears exactly once,
// each optional one at most once, features match, and every other pairing has
// a zero on one side.  The exact split (order 4) must hold all three offset
// pieces.  Segments may not overlap.

struct HxSlot {
  int kind = SEG_END, piece = 0, feat = 0;
  bool clash = false;
};

constexpr HxSlot hx_slot(const HxChunk& c, int slot) {
  HxSlot out;
  for (int k = 0; k < HX_SEGS; ++k) {
    const HxSeg& g = c.s[k];
    if (g.kind == SEG_END) break;
    if (g.slot + g.cap > 32) out.clash = true;
    if (slot < g.slot || slot >= g.slot + g.cap) continue;
    if (out.kind != SEG_END) out.clash = true;
    const int off = slot - g.slot;
    out.kind = g.kind;
    out.piece = g.kind == SEG_A ? g.piece + off : g.piece;
    out.feat = g.foff + off;
  }
  return out;
}

constexpr bool hx_valid(const HxRecipe& R) {
  int cnt[64][4][4] = {};
  int ai[4] = {}, aj[4] = {};
  if (R.nm < 1 || R.nm > HX_MFMAS || R.nc > HX_CHUNKS || R.nb > HX_CHUNKS) return false;
  if (R.order != 3 && R.order != 4) return false;
  for (int m = 0; m < R.nm; ++m) {
    if (R.sa[m] < 0 || R.sa[m] >= R.nc || R.sb[m] < 0 || R.sb[m] >= R.nb) return false;
    for (int slot = 0; slot < 32; ++slot) {
      const HxSlot c = hx_slot(R.col.ch[R.sa[m]], slot);
      const HxSlot r = hx_slot(R.row.ch[R.sb[m]], slot);
      if (c.clash || r.clash) return false;
      if (c.kind == SEG_END || r.kind == SEG_END) continue;
      if (c.kind == SEG_X && r.kind == SEG_X) {
        if (c.feat != r.feat || c.feat >= 64 || c.piece + r.piece > 4) return false;
        ++cnt[c.feat][c.piece][r.piece];
      } else if (c.kind == SEG_ONES && r.kind == SEG_A) {
        if (r.piece < 1 || r.piece > 3) return false;
        ++ai[r.piece];
      } else if (c.kind == SEG_A && r.kind == SEG_ONES) {
        if (c.piece < 1 || c.piece > 3) return false;
        ++aj[c.piece];
      } else {
        return false;
      }
    }
  }
  for (int k = 1; k <= 3; ++k) {
    const bool need = k <= 2 || R.order == 4;
    if (ai[k] > 1 || aj[k] > 1 || (need && (ai[k] != 1 || aj[k] != 1))) return false;
  }
  for (int f = 0; f < 64; ++f)
    for (int p = 1; p <= 3; ++p)
      for (int q = 1; q <= 3; ++q) {
        const bool real = f < R.maxd && p + q <= 4;
        const bool need = f < R.maxd && p + q <= R.order;
        if (cnt[f][p][q] > (real ? 1 : 0) || (need && cnt[f][p][q] != 1)) return false;
      }
  return true;
}

static_assert(hx_valid(HX_TABLE[0]) && hx_valid(HX_TABLE[1]) && hx_valid(HX_TABLE[2]) &&
                  hx_valid(HX_TABLE[3]) && hx_valid(HX_TABLE[4]) && hx_valid(HX_TABLE[5]) &&
                  hx_valid(HX_TABLE[6]),
              "a split-exponent recipe does not contract the intended sum");

template <int RID>
struct Hx {
  static constexpr int nc = HX_TABLE[RID].nc;
  static constexpr int nb = HX_TABLE[RID].nb;
  static constexpr int nm = HX_TABLE[RID].nm;
};

// Minimum waves per SIMD asked of the compiler.  At 2 a wave has at most 256
// registers and the matrix instructions then accumulate in ordinary VGPRs, so
// the vector ALUs read the exponent tiles without copies out of the
// accumulation registers.  The variants listed take 1 (accumulation
// registers, up to 512 per wave): their operands and accumulators do not fit
// in 256 registers (they spill at 2, checked per instantiation).  Moving the
// others to 2 left the results bitwise equal and took 7-23% off the products
// at b = 48 (D <= 30), b = 64 (D <= 8) and D > 32 (b <= 32).
template <int RID, int NCB, int NIB>
constexpr int hx_waves() {
  const bool big = (NIB == 2 && RID == 6 && NCB == 4) ||
                   (NIB == 4 && ((NCB == 4 && RID >= 2) || (NCB == 3 && RID >= 4) ||
                                 (NCB == 2 && RID >= 6))) ||
                   (NIB == 8 && NCB >= 2 && RID >= 2);
  return big ? 1 : 2;
}

// Waves per SIMD for the symmetric row sums: two wherever the variant fits
// 256 registers, so its matrix instructions accumulate in VGPRs and the
// exponent tiles reach the vector ALUs without v_accvgpr_read copies (one per
// value: about a seventh of the pass's instructions at D <= 30, 8 row tiles).
// The widest layouts with 8 row tiles would spill there and keep one wave.
template <int RID, int NIB, bool SQ>
constexpr int hx_sym_waves() {
  return (NIB == 8 && (RID >= 5 || (RID == 4 && SQ))) ? 1 : 2;
}
// The same for the plain row sums (rectangular sums, one right-hand side):
// only the widest layout with 8 row tiles would spill.
template <int RID, int NIB>
constexpr int hx_plain_waves() {
  return (NIB == 8 && RID >= 6) ? 1 : 2;
}

// ------------------------------------------------------------------ packing
//
// One thread per (padded) point computes the three float16 pieces of each
// coordinate (scaled) and of the offset once, and writes all of the point's
// slots, whose contents are resolved at compile time from the recipe.
// `scale` multiplies the coordinates (s on the column side, 2 beta log2(e) / s
// on the row side); the offset is neg_bl ||x||^2 + shift with
// neg_bl = -beta log2(e), in float64.  Padded points have zero coordinates and
// offset -65504, so their kernel values are 0.
template <int RID, bool ROW>
constexpr const HxSide& hx_side() {
  return ROW ? HX_TABLE[RID].row : HX_TABLE[RID].col;
}

// The pieces of v: each the float16 nearest to (the float32 rounding of) what
// the earlier ones leave; each remainder is exact in float64.  The float32
// step is kept explicit (an empty statement on the value): folded into one
// float64 -> float16 rounding, the conversion has no instruction on gfx950 and
// becomes a long integer sequence.
__device__ __forceinline__ void pieces3(double v, float (&out)[3]) {
  v = fmin(fmax(v, -65504.0), 65504.0);
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    float vf = float(v);
    asm volatile("" : "+v"(vf));
    const float h = float(_Float16(vf));
    out[q] = h;
    v -= double(h);
  }
}

// value of slot S = 32 ch + 8 g + e of the point
template <int RID, bool ROW, int S, int M>
__device__ __forceinline__ _Float16 hx_slot_value(const float (&px)[M][3], const float (&pa)[3]) {
  constexpr HxSlot v = hx_slot(hx_side<RID, ROW>().ch[S / 32], S % 32);
  if constexpr (v.kind == SEG_X && v.feat < M && v.piece >= 1 && v.piece <= 3)
    return _Float16(px[v.feat][v.piece - 1]);
  else if constexpr (v.kind == SEG_ONES)
    return _Float16(1.f);
  else if constexpr (v.kind == SEG_A && v.piece >= 1 && v.piece <= 3)
    return _Float16(pa[v.piece - 1]);
  else
    return _Float16(0.f);
}

// lane (g, p) word of chunk ch, for CG = 4 ch + g = 0 .. 4 nch - 1
template <int RID, bool ROW, int NCH, int M, int CG = 0>
__device__ __forceinline__ void hx_emit(const float (&px)[M][3], const float (&pa)[3],
                                        uintx4* __restrict__ out, int64_t tile, int p) {
  if constexpr (CG < 4 * NCH) {
    constexpr int CH = CG / 4, G = CG % 4, S = 32 * CH + 8 * G;
    halfx8 h;
    h[0] = hx_slot_value<RID, ROW, S + 0, M>(px, pa);
    h[1] = hx_slot_value<RID, ROW, S + 1, M>(px, pa);
    h[2] = hx_slot_value<RID, ROW, S + 2, M>(px, pa);
    h[3] = hx_slot_value<RID, ROW, S + 3, M>(px, pa);
    h[4] = hx_slot_value<RID, ROW, S + 4, M>(px, pa);
    h[5] = hx_slot_value<RID, ROW, S + 5, M>(px, pa);
    h[6] = hx_slot_value<RID, ROW, S + 6, M>(px, pa);
    h[7] = hx_slot_value<RID, ROW, S + 7, M>(px, pa);
    out[(tile * NCH + CH) * 64 + 16 * G + p] = __builtin_bit_cast(uintx4, h);
    hx_emit<RID, ROW, NCH, M, CG + 1>(px, pa, out, tile, p);
  }
}

template <int RID, bool ROW>
__global__ __launch_bounds__(256) void pack_hx_point_kernel(const float* __restrict__ X, int64_t n,
                                                            int D, int64_t ldx, double scale,
                                                            double neg_bl, double shift,
                                                            int64_t npad,
                                                            uintx4* __restrict__ out,
                                                            const double* __restrict__ mu,
                                                            HxGate gate) {
  constexpr int M = HX_TABLE[RID].maxd;
  constexpr int NCH = ROW ? HX_TABLE[RID].nb : HX_TABLE[RID].nc;
  if (hx_gate_closed(gate)) return;
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= npad) return;
  const bool real = i < n;
  const float* xi = X + min(i, n - 1) * ldx;
  float xv[M];
#pragma unroll
  for (int f = 0; f < M; ++f) xv[f] = xi[min(f, D - 1)];
  float px[M][3];
  double r = 0.0;
#pragma unroll
  for (int f = 0; f < M; ++f) {
    const bool use = real && f < D;
    // centred on mu in float64 (translation invariance of the kernel)
    const double v = use ? double(xv[f]) - (mu != nullptr ? mu[min(f, D - 1)] : 0.0) : 0.0;
    r += v * v;
    pieces3(scale * v, px[f]);
  }
  float pa[3];
  pieces3(real ? neg_bl * r + shift : -65504.0, pa);
  hx_emit<RID, ROW, NCH, M>(px, pa, out, i / TILE, int(i % TILE));
}

// ------------------------------------------------------------------ exponent

// t += sum over the recipe's instructions M.. of column chunk x row chunk.
template <int RID, int M = 0>
__device__ __forceinline__ void hx_chain(floatx4& t, const uintx4* xa, const uintx4* br) {
  if constexpr (M < HX_TABLE[RID].nm) {
    constexpr int ca = HX_TABLE[RID].sa[M];
    constexpr int cb = HX_TABLE[RID].sb[M];
    t = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, xa[ca]),
                                               __builtin_bit_cast(halfx8, br[cb]), t, 0, 0, 0);
    hx_chain<RID, M + 1>(t, xa, br);
  }
}

// Shift of the exponents: K' = 2^SHIFT K.
constexpr float SHIFT = 15.f;

// Exponent tile T^T[4g + r][p] of one row tile against one column tile (the
// shift included); DIAG: the same 16 points on both sides, entry j == i set
// to its exact value SHIFT.
template <int RID, bool DIAG>
__device__ __forceinline__ floatx4 hx_exponent(const uintx4* xa, const uintx4* br, int g, int p) {
  floatx4 t = floatx4{0.f, 0.f, 0.f, 0.f};
  hx_chain<RID>(t, xa, br);
  if (DIAG) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (4 * g + r == p) t[r] = SHIFT;
  }
  return t;
}

// ------------------------------------------------------------------ product

template <int RID, int NCB>
struct HxPair {
  uintx4 xa[2][Hx<RID>::nc];
  VSplit v[NCB];
};

template <int RID, int NCB>
__device__ __forceinline__ void load_hx_pair(HxPair<RID, NCB>& c, const uintx4* __restrict__ xc,
                                             const VSplit* __restrict__ vp, int64_t jp,
                                             int lane) {
  constexpr int NC = Hx<RID>::nc;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int64_t jb = 2 * jp + t;
#pragma unroll
    for (int ch = 0; ch < NC; ++ch) c.xa[t][ch] = xc[(jb * NC + ch) * 64 + lane];
  }
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) c.v[cb] = vp[(jp * NCB + cb) * 64 + lane];
}

// One pair of column tiles against the wave's NIB row tiles.  From the two
// exponent tiles lane (g, p) holds K'[p][J0 + 4g + r] and K'[p][J1 + 4g + r],
// which are its eight A-operand values (k = 8g + e, e = r for J0 and 4 + r for
// J1) of the K*V instruction; the V pack stores the matching rows per lane.
template <int RID, int NCB, int NIB, bool DIAG>
__device__ __forceinline__ void hx_pair(const HxPair<RID, NCB>& c,
                                        const uintx4 (&br)[NIB][Hx<RID>::nb],
                                        floatx4 (&acc)[NIB][NCB], int64_t jp, int64_t ib0,
                                        float m1, int g, int p) {
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
    floatx4 t[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (DIAG && 2 * jp + u == ib0 + ib)
        t[u] = hx_exponent<RID, true>(c.xa[u], br[ib], g, p);
      else
        t[u] = hx_exponent<RID, false>(c.xa[u], br[ib], g, p);
    }
    uintx4 hw, lw;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 4; r += 2) {
        // K' = 2^t with the shift in t: K' <= 2^15 (up to rounding)
        const float k0 = __builtin_amdgcn_exp2f(t[u][r]);
        const float k1 = __builtin_amdgcn_exp2f(t[u][r + 1]);
        unsigned hh, ll;
        split2m(k0, k1, m1, hh, ll);
        hw[2 * u + r / 2] = hh;
        lw[2 * u + r / 2] = ll;
      }
    const halfx8 khi = __builtin_bit_cast(halfx8, hw);
    const halfx8 klo = __builtin_bit_cast(halfx8, lw);
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      acc[ib][cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(khi, c.v[cb].hi, acc[ib][cb], 0, 0, 0);
      acc[ib][cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(khi, c.v[cb].lo, acc[ib][cb], 0, 0, 0);
      acc[ib][cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(klo, c.v[cb].hi, acc[ib][cb], 0, 0, 0);
    }
  }
  // one matrix instruction, then its share of the exponentials and three
  // other vector instructions (3.5% faster at D = 30, b = 32; unchanged at
  // D = 12, b = 16)
  sched_interleave<NIB * (2 * Hx<RID>::nm + 3 * NCB), 8 * NIB, 3>();
}

// One workgroup = 4 waves; wave w owns row tiles [ib0, ib0 + NIB).  The
// workgroup's column split is streamed in pairs of tiles through two operand
// buffers used in turn: a buffer is refilled right after its pair is
// consumed, so each load has a whole pair's compute to land.  Chunk totals of
// the two-level sum live in LDS, which keeps registers free for more waves.
// m1 = -1 (see split2m).
template <int RID, int NCB, int NIB>
__global__ __launch_bounds__(WG_THREADS)
__attribute__((amdgpu_waves_per_eu(hx_waves<RID, NCB, NIB>()))) void product_hx_kernel(
    const uintx4* __restrict__ xc, const VSplit* __restrict__ vp, const uintx4* __restrict__ xr,
    int64_t nrt, int64_t njp, int64_t jp_per_split, int diag, float m1,
    const float* __restrict__ colscale, const float* __restrict__ sl, float* __restrict__ Y,
    int64_t ldy, int64_t Nr, int b, float* __restrict__ part, int64_t nrpad, HxGate gate) {
  constexpr int NB = Hx<RID>::nb;
  __shared__ floatx4 tot[4][NIB][NCB][64];
  if (hx_gate_closed(gate)) return;
  const int lane = threadIdx.x & 63;
  // the wave index is uniform: make the row-tile range (and the diagonal
  // tests on it) scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t split = wr / nrt;
  const int64_t rt = wr % nrt;
  const int64_t ib0 = (rt * 4 + wave) * NIB;
  const int64_t jp_begin = split * jp_per_split;
  const int64_t jp_end = min(njp, jp_begin + jp_per_split);
  const int g = lane >> 4, p = lane & 15;

  uintx4 br[NIB][NB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
    for (int ch = 0; ch < NB; ++ch) br[ib][ch] = xr[((ib0 + ib) * NB + ch) * 64 + lane];
  floatx4 acc[NIB][NCB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      acc[ib][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
      tot[wave][ib][cb][lane] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

  auto step = [&](const HxPair<RID, NCB>& c, int64_t jp) {
    if (diag && 2 * jp + 1 >= ib0 && 2 * jp < ib0 + NIB)
      hx_pair<RID, NCB, NIB, true>(c, br, acc, jp, ib0, m1, g, p);
    else
      hx_pair<RID, NCB, NIB, false>(c, br, acc, jp, ib0, m1, g, p);
  };
  HxPair<RID, NCB> b0, b1;
  load_hx_pair(b0, xc, vp, jp_begin, lane);
  // keep b0's loads ahead of b1's, the order the loop keeps them in: the wait
  // before each step then only covers the buffer it consumes
  __builtin_amdgcn_sched_barrier(0);
  load_hx_pair(b1, xc, vp, min(jp_begin + 1, jp_end - 1), lane);
  int chunk = 0;
  for (int64_t jp = jp_begin; jp < jp_end; jp += 2) {
    step(b0, jp);
    load_hx_pair(b0, xc, vp, min(jp + 2, jp_end - 1), lane);
    // the refill is unconditional (clamped index) so that the number of loads
    // in flight at the top of the loop is the same on every path
    if (jp + 1 < jp_end) step(b1, jp + 1);
    load_hx_pair(b1, xc, vp, min(jp + 3, jp_end - 1), lane);
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

// ------------------------------------------------------------------ row sums

template <int RID>
struct HxCol {
  uintx4 xa[Hx<RID>::nc];
  floatx4 w;
};

template <int RID, bool UNIT>
__device__ __forceinline__ void load_hx_col(HxCol<RID>& c, const uintx4* __restrict__ xc,
                                            const floatx4* __restrict__ wp, int64_t jb,
                                            int lane) {
  constexpr int NC = Hx<RID>::nc;
#pragma unroll
  for (int ch = 0; ch < NC; ++ch) c.xa[ch] = xc[(jb * NC + ch) * 64 + lane];
  if (!UNIT) c.w = wp[jb * 64 + lane];
}

// One column tile against the wave's NIB row tiles: all exponent chains
// first (independent chains issue back to back and the exponentials can
// overlap their tail), then K' = 2^t summed (times the weights) on the vector
// ALUs.
template <int RID, int NIB, bool UNIT, bool DIAG, bool SQ = false>
__device__ __forceinline__ void hx_rowsum_tile(const HxCol<RID>& c,
                                               const uintx4 (&br)[NIB][Hx<RID>::nb],
                                               float (&acc)[NIB], int64_t jb, int64_t ib0, int g,
                                               int p, float (*acc2)[NIB] = nullptr) {
  floatx4 t[NIB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
    if (DIAG && jb == ib0 + ib)
      t[ib] = hx_exponent<RID, true>(c.xa, br[ib], g, p);
    else
      t[ib] = hx_exponent<RID, false>(c.xa, br[ib], g, p);
  }
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
    float k[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) k[r] = __builtin_amdgcn_exp2f(t[ib][r]);
    if (UNIT) {
      acc[ib] += (k[0] + k[1]) + (k[2] + k[3]);
    } else {
      // one FMA per entry: as many vector instructions as the unit-weight sum
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[ib] = fmaf(k[r], c.w[r], acc[ib]);
    }
    if constexpr (SQ) {
      // (K')^2 = 2^30 K^2: the kernel at twice the bandwidth, unit weights
#pragma unroll
      for (int r = 0; r < 4; ++r) (*acc2)[ib] = fmaf(k[r], k[r], (*acc2)[ib]);
    }
  }
}

// Row sums sum_j K_ij w_j (b = 1, the normalisation passes): the same
// exponent tiles, reduced on the vector ALUs instead of a second contraction.
// Column tiles stream through two operand buffers used in turn.
template <int RID, int NIB, bool UNIT>
__global__ __launch_bounds__(WG_THREADS)
__attribute__((amdgpu_waves_per_eu(hx_plain_waves<RID, NIB>()))) void rowsum_hx_kernel(
    const uintx4* __restrict__ xc, const floatx4* __restrict__ wp, const uintx4* __restrict__ xr,
    int64_t nrt, int64_t njb, int64_t jb_per_split, int diag, float* __restrict__ out,
    int64_t Nr, float* __restrict__ part, int64_t nrpad, HxGate gate) {
  constexpr int NB = Hx<RID>::nb;
  if (hx_gate_closed(gate)) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t split = wr / nrt;
  const int64_t rt = wr % nrt;
  const int64_t ib0 = (rt * 4 + wave) * NIB;
  const int64_t jb_begin = split * jb_per_split;
  const int64_t jb_end = min(njb, jb_begin + jb_per_split);
  const int g = lane >> 4, p = lane & 15;

  uintx4 br[NIB][NB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
    for (int ch = 0; ch < NB; ++ch) br[ib][ch] = xr[((ib0 + ib) * NB + ch) * 64 + lane];
  float acc[NIB], tot[NIB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) acc[ib] = tot[ib] = 0.f;

  auto step = [&](const HxCol<RID>& c, int64_t jb) {
    if (diag && jb >= ib0 && jb < ib0 + NIB)
      hx_rowsum_tile<RID, NIB, UNIT, true>(c, br, acc, jb, ib0, g, p);
    else
      hx_rowsum_tile<RID, NIB, UNIT, false>(c, br, acc, jb, ib0, g, p);
  };
  HxCol<RID> b0, b1;
  b0.w = b1.w = floatx4{1.f, 1.f, 1.f, 1.f};
  load_hx_col<RID, UNIT>(b0, xc, wp, jb_begin, lane);
  __builtin_amdgcn_sched_barrier(0);  // b0's loads ahead of b1's, as in the loop
  load_hx_col<RID, UNIT>(b1, xc, wp, min(jb_begin + 1, jb_end - 1), lane);
  int chunk = 0;
  for (int64_t jb = jb_begin; jb < jb_end; jb += 2) {
    step(b0, jb);
    load_hx_col<RID, UNIT>(b0, xc, wp, min(jb + 2, jb_end - 1), lane);
    if (jb + 1 < jb_end) step(b1, jb + 1);
    load_hx_col<RID, UNIT>(b1, xc, wp, min(jb + 3, jb_end - 1), lane);
    chunk += 2;
    if (chunk >= CHUNK_TILES) {
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
    // undo the shift (exact) and add the four lanes p, p+16, p+32, p+48 of row p
    float v = (tot[ib] + acc[ib]) * 0x1p-15f;
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

// ------------------------------------------------------------------ symmetric row sums
//
// When rows and columns are the same N points, K is symmetric and each
// off-diagonal tile K_IJ can serve both sums: q_I += K_IJ w_J along its rows and
// q_J += K_IJ^T w_I along its columns, so every kernel entry off the diagonal
// blocks is evaluated (and exponentiated) once instead of twice.
//
// Points are grouped in blocks of 512 (one workgroup's 4 waves x 8 row tiles);
// with B blocks and h = (B - 1) / 2, the workgroup of block P takes its own
// block (row sums only, exact diagonal) and then the blocks P + 1 .. P + h
// (mod B), plus P + B/2 when B is even and P < B/2: every unordered pair of
// distinct blocks is then taken exactly once.  That column range is split over
// nsplit workgroups.  Row sums go to per-split partials as in the plain kernel.
// Column sums are reduced over the wave's 128 rows (in-lane over its row
// tiles, then across the 16 lanes of a DPP row), converted to 64-bit fixed
// point and added into a per-workgroup LDS array with integer LDS atomics; every
// SYM_CHUNK column tiles the workgroup adds that array into the global
// per-point accumulator with integer atomics.  Integer addition is exact and
// order-free, so the result is bitwise reproducible.  (Global atomics inside
// the tile loop would make each operand-load wait also wait for an atomic's
// round trip, since vector memory operations retire in order.)  The
// fixed-point scale assumes weights in [0, 1] (the normalisation weights
// q^-alpha with q >= 1 are) and leaves a factor 4 of headroom below 2^63 for
// the total.

// Column tiles whose fixed-point column sums a workgroup gathers in LDS
// (SYM_CHUNK x 16 x 8 bytes) before adding them into global memory; even.
constexpr int SYM_CHUNK = 256;

// Sum of v over the 16 lanes of the lane's DPP row (every lane gets the sum).
__device__ __forceinline__ float dpp_row_sum(float v) {
  // xor 1 and xor 2 inside quads, then mirrored quads and mirrored half-rows
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1,
                                                             0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E,
                                                             0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x141,
                                                             0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x140,
                                                             0xF, 0xF, false));
  return v;
}

// One pipeline step of the symmetric row sums.  t holds the exponent tiles of
// an off-diagonal column tile J against the wave's NIB row tiles; each is
// exponentiated and then overwritten with the exponent tile of the next column
// tile (operands xn), so the matrix-core chain of row tile ib runs alongside
// the vector work of row tiles ib + 1, ...  SUMS: add J's row sums into acc and
// its column sums into the fixed-point accumulator (false for padding tiles).
template <int RID, int NIB, bool UNIT, bool SUMS, bool SQ>
__device__ __forceinline__ void hx_sym_step(floatx4 (&t)[NIB], const uintx4* xn,
                                            const uintx4 (&br)[NIB][Hx<RID>::nb],
                                            const floatx4& w, const float (&wi)[NIB],
                                            float (&acc)[NIB], float (&acc2)[NIB], int64_t jl,
                                            double fix_scale, double fix_scale2,
                                            unsigned long long* lds_col,
                                            unsigned long long* lds_col2, int g, int p) {
  float cs[4] = {0.f, 0.f, 0.f, 0.f};
  float cs2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
    float k[4];
    if (SUMS) {
#pragma unroll
      for (int r = 0; r < 4; ++r) k[r] = __builtin_amdgcn_exp2f(t[ib][r]);
    }
    t[ib] = hx_exponent<RID, false>(xn, br[ib], g, p);
    if (SUMS) {
      if (UNIT) {
        acc[ib] += (k[0] + k[1]) + (k[2] + k[3]);
#pragma unroll
        for (int r = 0; r < 4; ++r) cs[r] += k[r];
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          acc[ib] = fmaf(k[r], w[r], acc[ib]);
          cs[r] = fmaf(k[r], wi[ib], cs[r]);
        }
        if constexpr (SQ) {
          // the squared kernel (K at twice the bandwidth) with unit weights,
          // along the rows and along the columns of the tile
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            acc2[ib] = fmaf(k[r], k[r], acc2[ib]);
            cs2[r] = fmaf(k[r], k[r], cs2[r]);
          }
        }
      }
    }
  }
  if (!SUMS) return;
  // the row sums are due here (an empty statement reading them), not sunk
  // past the column-sum atomic below, so that they interleave too
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
    asm volatile("" ::"v"(acc[ib]));
    if constexpr (SQ) asm volatile("" ::"v"(acc2[ib]));
  }
  // Interleave the contraction with the exponentials and sums (left to
  // itself the scheduler issues the exponentials first, then the matrix
  // instructions with little vector work between them).
  sched_interleave<Hx<RID>::nm * NIB, 4 * NIB, SQ ? 5 : 3>();
  // lane (g, p) holds, for column 4g + r of the tile, the sum over rows p of
  // the wave's tiles; the 16 lanes of DPP row g hold the wave's other rows
#pragma unroll
  for (int r = 0; r < 4; ++r) cs[r] = dpp_row_sum(cs[r]);
  // lane p < 4 adds column 4g + p (selects, no branches)
  const float v01 = (p & 1) ? cs[1] : cs[0];
  const float v23 = (p & 1) ? cs[3] : cs[2];
  const float v = (p & 2) ? v23 : v01;
  const long long fx = __double2ll_rn(double(v) * fix_scale);
  if (p < 4) atomicAdd(lds_col + jl * TILE + 4 * g + p, static_cast<unsigned long long>(fx));
  if constexpr (SQ) {
#pragma unroll
    for (int r = 0; r < 4; ++r) cs2[r] = dpp_row_sum(cs2[r]);
    const float u01 = (p & 1) ? cs2[1] : cs2[0];
    const float u23 = (p & 1) ? cs2[3] : cs2[2];
    const float u = (p & 2) ? u23 : u01;
    const long long fx2 = __double2ll_rn(double(u) * fix_scale2);
    if (p < 4) atomicAdd(lds_col2 + jl * TILE + 4 * g + p, static_cast<unsigned long long>(fx2));
  }
}

// SQ (weighted passes only): also the row and column sums of the squared
// kernel, K^2 1 = K(2 beta) 1 (eq. kernel), into part2 / colfix2 with the scale
// fix_scale2 per unit of (2^15 K)^2.
template <int RID, int NIB, bool UNIT, bool SQ = false>
__global__ __launch_bounds__(WG_THREADS)
__attribute__((amdgpu_waves_per_eu(hx_sym_waves<RID, NIB, SQ>()))) void rowsum_sym_hx_kernel(
    const uintx4* __restrict__ xc, const floatx4* __restrict__ wp, const uintx4* __restrict__ xr,
    int64_t nblk, int64_t njb, int64_t jb_per_split, int64_t nsplit, float* __restrict__ part,
    int64_t nrpad, unsigned long long* __restrict__ colfix, double fix_scale,
    float* __restrict__ part2, unsigned long long* __restrict__ colfix2, double fix_scale2,
    HxGate gate) {
  static_assert(!(SQ && UNIT), "squared sums ride on a weighted pass");
  if (hx_gate_closed(gate)) return;
  constexpr int NB = Hx<RID>::nb;
  constexpr int NC = Hx<RID>::nc;
  constexpr int BT = 4 * NIB;  // tiles per block
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = xcd_remap(blockIdx.x, gridDim.x);
  // whole-block splits: number the workgroups by the block c their window
  // starts at (c = P + split * blocks per split), so that consecutive ids (run
  // together on one XCD) read the same column tiles
  const int64_t jbk = jb_per_split / BT;
  int64_t split, P;
  if (jb_per_split % BT == 0) {
    const int64_t c = wr / nsplit;
    split = wr % nsplit;
    P = ((c - split * jbk) % nblk + nblk) % nblk;
  } else {
    split = wr / nblk;
    P = wr % nblk;
  }
  const int64_t ib0 = P * BT + wave * NIB;
  const int64_t h = (nblk - 1) / 2;
  const int64_t span = BT * (1 + h + ((nblk % 2 == 0 && 2 * P < nblk) ? 1 : 0));
  const int64_t jj_begin = split * jb_per_split;
  const int64_t jj_end = min(span, jj_begin + jb_per_split);
  const int64_t ntile = nblk * BT;
  const int g = lane >> 4, p = lane & 15;
  // fixed-point column sums of the current chunk of SYM_CHUNK tiles
  __shared__ unsigned long long lds_col[SYM_CHUNK * TILE];
  __shared__ unsigned long long lds_col2[SQ ? SYM_CHUNK * TILE : 1];
  for (int e = threadIdx.x; e < SYM_CHUNK * TILE; e += WG_THREADS) {
    lds_col[e] = 0ull;
    if constexpr (SQ) lds_col2[e] = 0ull;
  }
  __syncthreads();

  uintx4 br[NIB][NB];
  float wi[NIB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
    for (int ch = 0; ch < NB; ++ch) br[ib][ch] = xr[((ib0 + ib) * NB + ch) * 64 + lane];
    // weight of own row 16 (ib0 + ib) + p: pack element (tile, lane 16 (p / 4), p % 4);
    // own tiles past the column pack are padding rows (their kernel values are 0)
    wi[ib] = 0.f;
    if (!UNIT && ib0 + ib < njb)
      wi[ib] = reinterpret_cast<const float*>(wp)[((ib0 + ib) * 64 + 16 * (p >> 2)) * 4 + (p & 3)];
  }
  float acc[NIB], tot[NIB], acc2[NIB], tot2[NIB];
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) acc[ib] = tot[ib] = acc2[ib] = tot2[ib] = 0.f;

  // column tile of range position jj (0 <= jj < span <= ntile + BT, cyclic over
  // the blocks); -1 for the padding tiles past the real columns
  const int base = int(P * BT), nt32 = int(ntile), njb32 = int(njb);
  auto tile_of = [&](int64_t jj) -> int {
    int J = base + int(jj);
    if (J >= nt32) J -= nt32;
    return J < njb32 ? J : -1;
  };
  // tile loaded for range position jj of [lo, jj_end): clamped into the range,
  // padding tiles read tile 0, so that loads are unconditional and every path
  // keeps the same loads in flight
  auto load_tile = [&](int64_t jj, int64_t lo) -> int64_t {
    const int J = tile_of(max(min(jj, jj_end - 1), lo));
    return J < 0 ? 0 : J;
  };
  int chunk = 0;
  auto row_chunk = [&](int tiles) {
    chunk += tiles;
    if (chunk >= CHUNK_TILES) {
      chunk = 0;
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) {
        tot[ib] += acc[ib];
        acc[ib] = 0.f;
        if constexpr (SQ) {
          tot2[ib] += acc2[ib];
          acc2[ib] = 0.f;
        }
      }
    }
  };

  // The workgroup's own block (range positions below BT, in split 0 only):
  // plain row sums, exact diagonal.  Column tiles stream through two buffers
  // used in turn.
  const int64_t own_end = min(jj_end, int64_t(BT));
  if (jj_begin < own_end) {
    auto step = [&](const HxCol<RID>& c, int64_t jj) {
      const int J = tile_of(jj);
      if (J < 0) return;
      if (J >= ib0 && J < ib0 + NIB)
        hx_rowsum_tile<RID, NIB, UNIT, true, SQ>(c, br, acc, J, ib0, g, p, &acc2);
      else
        hx_rowsum_tile<RID, NIB, UNIT, false, SQ>(c, br, acc, J, ib0, g, p, &acc2);
    };
    HxCol<RID> b0, b1;
    b0.w = b1.w = floatx4{1.f, 1.f, 1.f, 1.f};
    load_hx_col<RID, UNIT>(b0, xc, wp, load_tile(jj_begin, jj_begin), lane);
    __builtin_amdgcn_sched_barrier(0);  // b0's loads ahead of b1's, as in the loop
    load_hx_col<RID, UNIT>(b1, xc, wp, load_tile(min(jj_begin + 1, own_end - 1), jj_begin),
                           lane);
    for (int64_t jj = jj_begin; jj < own_end; jj += 2) {
      step(b0, jj);
      load_hx_col<RID, UNIT>(b0, xc, wp, load_tile(min(jj + 2, own_end - 1), jj_begin), lane);
      if (jj + 1 < own_end) step(b1, jj + 1);
      load_hx_col<RID, UNIT>(b1, xc, wp, load_tile(min(jj + 3, own_end - 1), jj_begin), lane);
      row_chunk(2);
    }
  }

  // The other blocks: each tile serves both sums.  Two-stage pipeline over
  // the tiles u = 0, 1, ... of [s0, jj_end): step u exponentiates and sums
  // tile u, whose exponents the previous step made, while the matrix cores
  // make those of tile u + 1 (hx_sym_step).  Tile v's column operands sit in
  // slot v % 2 and are loaded two steps ahead of their contraction, its
  // weights one step ahead of its sums.
  const int64_t s0 = max(jj_begin, int64_t(BT));
  const int64_t n2 = jj_end - s0;
  if (n2 > 0) {
    uintx4 xa[2][NC];
    floatx4 w[2];
    floatx4 t[NIB];
    w[0] = w[1] = floatx4{1.f, 1.f, 1.f, 1.f};
    auto load_xa = [&](uintx4 (&dst)[NC], int64_t u) {
      const int64_t J = load_tile(s0 + u, s0);
#pragma unroll
      for (int ch = 0; ch < NC; ++ch) dst[ch] = xc[(J * NC + ch) * 64 + lane];
    };
    auto load_w = [&](floatx4& dst, int64_t u) {
      if (!UNIT) dst = wp[load_tile(s0 + u, s0) * 64 + lane];
    };
    load_xa(xa[0], 0);
    load_w(w[0], 0);
    __builtin_amdgcn_sched_barrier(0);
    load_xa(xa[1], 1);
    // consume the row operands here (an empty statement reading them): their
    // loads complete before the loop, whose waits then only ever cover the
    // column operands a step consumes (left to itself the compiler sinks these
    // loads past the loop entry and every iteration waits for all loads)
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
      for (int ch = 0; ch < NB; ++ch) asm volatile("" ::"v"(br[ib][ch]));
    // likewise the scalar kernel argument used in the loop: with its load done
    // here, the loop's LDS atomics (which share the counter) are never waited on
    asm volatile("" ::"s"(fix_scale));
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) t[ib] = hx_exponent<RID, false>(xa[0], br[ib], g, p);
    // step u (slot S = u % 2): operands of tile u + 2 into slot S, weights of
    // tile u + 1 into slot S ^ 1, sums of tile u with weights from slot S,
    // contraction of tile u + 1 from slot S ^ 1
    auto pipe_step = [&](auto S_, int64_t u) {
      constexpr int S = decltype(S_)::value;
      load_xa(xa[S], u + 2);
      load_w(w[S ^ 1], u + 1);
      const int J = tile_of(s0 + u);
      const int64_t jl = (s0 + u - jj_begin) % SYM_CHUNK;
      if (J >= 0)
        hx_sym_step<RID, NIB, UNIT, true, SQ>(t, xa[S ^ 1], br, w[S], wi, acc, acc2, jl,
                                              fix_scale, fix_scale2, lds_col, lds_col2, g, p);
      else
        hx_sym_step<RID, NIB, UNIT, false, SQ>(t, xa[S ^ 1], br, w[S], wi, acc, acc2, jl,
                                               fix_scale, fix_scale2, lds_col, lds_col2, g, p);
      row_chunk(1);
      // end of a chunk of column tiles (the trip count is uniform over the
      // workgroup): add the chunk's column sums into the global accumulator
      const int64_t done = s0 + u + 1 - jj_begin;
      if (done % SYM_CHUNK == 0 || s0 + u + 1 >= jj_end) {
        const int64_t c0 = jj_begin + (done - 1) / SYM_CHUNK * SYM_CHUNK;
        __syncthreads();
        for (int e = threadIdx.x; e < SYM_CHUNK * TILE; e += WG_THREADS) {
          const unsigned long long v = lds_col[e];
          const int Jc = c0 + e / TILE < jj_end ? tile_of(c0 + e / TILE) : -1;
          if (v != 0ull && Jc >= 0) atomicAdd(colfix + int64_t(Jc) * TILE + e % TILE, v);
          lds_col[e] = 0ull;
          if constexpr (SQ) {
            const unsigned long long v2 = lds_col2[e];
            if (v2 != 0ull && Jc >= 0) atomicAdd(colfix2 + int64_t(Jc) * TILE + e % TILE, v2);
            lds_col2[e] = 0ull;
          }
        }
        __syncthreads();
      }
    };
    for (int64_t u = 0; u < n2; u += 2) {
      pipe_step(std::integral_constant<int, 0>{}, u);
      if (u + 1 < n2) pipe_step(std::integral_constant<int, 1>{}, u + 1);
    }
  }
#pragma unroll
  for (int ib = 0; ib < NIB; ++ib) {
    float v = (tot[ib] + acc[ib]) * 0x1p-15f;
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (g == 0) part[split * nrpad + (ib0 + ib) * TILE + p] = v;
    if constexpr (SQ) {
      float v2 = (tot2[ib] + acc2[ib]) * 0x1p-30f;
      v2 += __shfl_xor(v2, 16);
      v2 += __shfl_xor(v2, 32);
      if (g == 0) part2[split * nrpad + (ib0 + ib) * TILE + p] = v2;
    }
  }
}

// ------------------------------------------------------------------ host dispatch

template <int RID, int NCB, int NIB>
void product_hx_launch(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                       const float* vp, const float* colscale, bool diag, const float* sl,
                       float* Y, int64_t ldy, int b, float* part, hipStream_t stream) {
  const unsigned grid = unsigned(p.nrt * p.nsplit);
  hipLaunchKernelGGL((product_hx_kernel<RID, NCB, NIB>), dim3(grid), dim3(WG_THREADS), 0, stream,
                     reinterpret_cast<const uintx4*>(cols.xp.p),
                     reinterpret_cast<const VSplit*>(vp),
                     reinterpret_cast<const uintx4*>(rows.xp.p), p.nrt, ceil_div(p.njb, 2),
                     p.jb_per_split / 2, int(diag), -1.0f, colscale, sl, Y, ldy, rows.n, b, part,
                     rows.npad, gate_of(rows));
  FD_LAUNCH_CHECK();
}

template <int RID, int NCB>
void product_hx_nib(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                    const float* vp, const float* cs, bool diag, const float* sl, float* Y,
                    int64_t ldy, int b, float* part, hipStream_t stream) {
  switch (p.nib) {
    case 2: return product_hx_launch<RID, NCB, 2>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
    case 4: return product_hx_launch<RID, NCB, 4>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
    case 8:
      if constexpr (RID <= 3 && NCB <= 2)
        return product_hx_launch<RID, NCB, 8>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
      break;
  }
  throw Error{FD_ERR_INVALID_ARG, "internal: unsupported rows per wave"};
}

template <int RID>
void product_hx_ncb(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                    const float* vp, const float* cs, bool diag, const float* sl, float* Y,
                    int64_t ldy, int b, float* part, hipStream_t stream) {
  switch (p.ncb) {
    case 1: return product_hx_nib<RID, 1>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
    case 2: return product_hx_nib<RID, 2>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
    case 3: return product_hx_nib<RID, 3>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
    case 4: return product_hx_nib<RID, 4>(p, rows, cols, vp, cs, diag, sl, Y, ldy, b, part, stream);
  }
  throw Error{FD_ERR_UNSUPPORTED, "block width above 64"};
}

template <int RID, int NIB, bool UNIT>
void rowsum_hx_launch(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                      const float* wp, bool diag, float* out, float* part, hipStream_t stream) {
  const unsigned grid = unsigned(p.nrt * p.nsplit);
  hipLaunchKernelGGL((rowsum_hx_kernel<RID, NIB, UNIT>), dim3(grid), dim3(WG_THREADS), 0, stream,
                     reinterpret_cast<const uintx4*>(cols.xp.p),
                     reinterpret_cast<const floatx4*>(wp),
                     reinterpret_cast<const uintx4*>(rows.xp.p), p.nrt, p.njb, p.jb_per_split,
                     int(diag), out, rows.n, part, rows.npad, gate_of(rows));
  FD_LAUNCH_CHECK();
}

template <int RID>
void rowsum_hx_u(const KVPlan& p, const PointPack& rows, const PointPack& cols, const float* wp,
                 bool diag, float* out, float* part, hipStream_t stream) {
  if (p.nib == 8) {
    if (wp == nullptr)
      rowsum_hx_launch<RID, 8, true>(p, rows, cols, wp, diag, out, part, stream);
    else
      rowsum_hx_launch<RID, 8, false>(p, rows, cols, wp, diag, out, part, stream);
    return;
  }
  if (wp == nullptr)
    rowsum_hx_launch<RID, 4, true>(p, rows, cols, wp, diag, out, part, stream);
  else
    rowsum_hx_launch<RID, 4, false>(p, rows, cols, wp, diag, out, part, stream);
}

template <int RID, int NIB, bool UNIT, bool SQ>
void rowsum_sym_hx_launch(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                          const float* wp, float* part, unsigned long long* colfix,
                          double fix_scale, const SymSquares& sq, hipStream_t stream) {
  const unsigned grid = unsigned(p.nrt * p.nsplit);
  hipLaunchKernelGGL((rowsum_sym_hx_kernel<RID, NIB, UNIT, SQ>), dim3(grid), dim3(WG_THREADS), 0,
                     stream, reinterpret_cast<const uintx4*>(cols.xp.p),
                     reinterpret_cast<const floatx4*>(wp),
                     reinterpret_cast<const uintx4*>(rows.xp.p), p.nrt, p.njb, p.jb_per_split,
                     int64_t(p.nsplit), part, rows.npad, colfix, fix_scale, sq.part, sq.colfix,
                     sq.fix_scale, gate_of(rows));
  FD_LAUNCH_CHECK();
}

template <int RID>
void rowsum_sym_hx_u(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                     const float* wp, float* part, unsigned long long* colfix, double fix_scale,
                     const SymSquares& sq, hipStream_t stream) {
  if (sq.part != nullptr) {
    // squared sums: weighted passes of the eight-tile plan only
    FD_REQUIRE(p.nib == 8 && wp != nullptr, FD_ERR_INVALID_ARG,
               "internal: squared sums need a weighted eight-tile pass");
    rowsum_sym_hx_launch<RID, 8, false, true>(p, rows, cols, wp, part, colfix, fix_scale, sq,
                                              stream);
    return;
  }
  if (p.nib == 4) {
    if (wp == nullptr)
      rowsum_sym_hx_launch<RID, 4, true, false>(p, rows, cols, wp, part, colfix, fix_scale, sq,
                                                stream);
    else
      rowsum_sym_hx_launch<RID, 4, false, false>(p, rows, cols, wp, part, colfix, fix_scale, sq,
                                                 stream);
    return;
  }
  if (wp == nullptr)
    rowsum_sym_hx_launch<RID, 8, true, false>(p, rows, cols, wp, part, colfix, fix_scale, sq,
                                              stream);
  else
    rowsum_sym_hx_launch<RID, 8, false, false>(p, rows, cols, wp, part, colfix, fix_scale, sq,
                                               stream);
}

void check_hx(const KVPlan& p, const PointPack& rows, const PointPack& cols) {
  FD_REQUIRE(rows.rid >= 0 && rows.rid < HX_RECIPES && rows.rid == cols.rid && rows.row_side &&
                 !cols.row_side,
             FD_ERR_INVALID_ARG, "internal: split packs do not match");
  const HxRecipe& R = HX_TABLE[rows.rid];
  const int64_t row_tiles = p.nrt * 4 * p.nib;
  check_span(rows.xp, size_t(row_tiles) * R.nb * 64 * 4, "split row pack");
  check_span(cols.xp, size_t(round_up(p.njb, 2)) * R.nc * 64 * 4, "split column pack");
}

}  // namespace

static_assert(HX_TABLE[4].order == 3 && HX_TABLE[6].order == 3 && HX_TABLE[4].maxd >= 30 &&
                  HX_TABLE[6].maxd >= 62,
              "full-offset recipes must serve the short recipes' feature widths");

int hx_recipe_for(int64_t D) {
  for (int r = 0; r < HX_RECIPES; ++r)
    if (D >= 1 && D <= HX_TABLE[r].maxd) return r;
  return -1;
}
// s = 2^e balances |x'| = s|x| and |b'| = 2 beta log2(e) |x| / s: both are
// then within a factor sqrt(2) of sqrt(2 beta log2(e)) |x|, at most 512 inside
// the exponent range, and neither falls towards float16's subnormals before
// the cross term itself is negligible.  (A clamp of e at +-12 made b' lose
// bits at beta < 2e-8 with large coordinates: 1.8e-5 K V error at B = 0.3.)
// |e| <= 64 only guards the float32 extremes of beta.
double hx_coord_scale(double beta) {
  int e = 0;
  if (beta > 0.0) e = std::clamp(int(std::lround(0.5 * std::log2(2.0 * beta * LOG2E))), -64, 64);
  return std::ldexp(1.0, e);
}

int hx_col_chunks(int rid) { return HX_TABLE[rid].nc; }
int hx_row_chunks(int rid) { return HX_TABLE[rid].nb; }

int hx_full_offset_recipe(int rid) {
  // short recipes that drop the third offset piece -> the next recipe up,
  // which keeps all three (checked at compile time below)
  return rid == 3 ? 4 : rid == 5 ? 6 : -1;
}

template <int RID, bool ROW>
static void pack_hx_launch(const float* X, int64_t n, int64_t D, int64_t ldx, double beta,
                           FSpan xp, int64_t npad, const double* mu, HxGate gate,
                           hipStream_t stream) {
  const HxRecipe& R = HX_TABLE[RID];
  const int nch = ROW ? R.nb : R.nc;
  check_span(xp, size_t(npad / TILE) * nch * 64 * 4, "split point pack");
  FD_REQUIRE(D <= R.maxd, FD_ERR_INVALID_ARG, "internal: recipe too narrow for D");
  const double bl = beta * LOG2E;
  const double s = hx_coord_scale(beta);
  const double scale = ROW ? 2.0 * bl / s : s;
  const double shift = ROW ? double(SHIFT) : 0.0;
  hipLaunchKernelGGL((pack_hx_point_kernel<RID, ROW>), dim3(blocks_for(npad, 256)), dim3(256), 0,
                     stream, X, n, int(D), ldx, scale, -bl, shift, npad,
                     reinterpret_cast<uintx4*>(xp.p), mu, gate);
  FD_LAUNCH_CHECK();
}

template <bool ROW>
static void pack_hx_rid(int rid, const float* X, int64_t n, int64_t D, int64_t ldx, double beta,
                        FSpan xp, int64_t npad, const double* mu, HxGate gate,
                        hipStream_t stream) {
  switch (rid) {
    case 0: return pack_hx_launch<0, ROW>(X, n, D, ldx, beta, xp, npad, mu, gate, stream);
    case 1: return pack_hx_launch<1, ROW>(X, n, D, ldx, beta, xp, npad, mu, gate, stream);
    case 2: return pack_hx_launch<2, ROW>(X, n, D, ldx, beta, xp, npad, mu, gate, stream);
    case 3: return pack_hx_launch<3, ROW>(X, n, D, ldx, beta, xp, npad, mu, gate, stream);
    case 4: return pack_hx_launch<4, ROW>(X, n, D, ldx, beta, xp, npad, mu, gate, stream);
    case 5: return pack_hx_launch<5, ROW>(X, n, D, ldx, beta, xp, npad, mu, gate, stream);
    case 6: return pack_hx_launch<6, ROW>(X, n, D, ldx, beta, xp, npad, mu, gate, stream);
  }
  throw Error{FD_ERR_UNSUPPORTED, "feature dimension above 64"};
}

void launch_pack_points_hx(const float* X, int64_t n, int64_t D, int64_t ldx, double beta,
                           bool row_side, PointPack& out, const CentreWs* centre,
                           hipStream_t stream) {
  const int rid = hx_recipe_for(D);
  FD_REQUIRE(rid >= 0, FD_ERR_UNSUPPORTED, "feature dimension above 64");
  FD_REQUIRE(out.npad % (2 * TILE) == 0 && out.npad >= n, FD_ERR_INVALID_ARG,
             "internal: bad split pack geometry");
  const double* mu = centre != nullptr ? centre->mu : nullptr;
  const int wide = centre != nullptr ? hx_full_offset_recipe(rid) : -1;
  out.rid = rid;
  out.row_side = row_side;
  out.rid2 = wide;
  out.variant = wide >= 0 ? 1 : 0;
  out.r2max = wide >= 0 ? centre->r2max : nullptr;
  const HxGate g1{out.r2max, beta * LOG2E, out.variant};
  if (row_side)
    pack_hx_rid<true>(rid, X, n, D, ldx, beta, out.xp, out.npad, mu, g1, stream);
  else
    pack_hx_rid<false>(rid, X, n, D, ldx, beta, out.xp, out.npad, mu, g1, stream);
  if (wide >= 0) {
    const HxGate g2{out.r2max, beta * LOG2E, 2};
    if (row_side)
      pack_hx_rid<true>(wide, X, n, D, ldx, beta, out.xp2, out.npad, mu, g2, stream);
    else
      pack_hx_rid<false>(wide, X, n, D, ldx, beta, out.xp2, out.npad, mu, g2, stream);
  }
}

// The second layout of a pack pair (see PointPack): same geometry, the
// full-offset recipe's chunks.
static PointPack full_offset_view(const PointPack& pk) {
  PointPack q = pk;
  q.xp = pk.xp2;
  q.rid = pk.rid2;
  q.variant = 2;
  return q;
}

// Runs `go` on the packs as filled and, when they hold both layouts, again on
// the full-offset one: each launch reads the exponent-budget word and only
// the matching one works.  The pair counts as one launch for the timing hooks.
template <class Go>
static void dual_dispatch(const PointPack& rows, const PointPack& cols, fd_kernel_kind kind,
                          hipStream_t stream, Go&& go) {
  FD_REQUIRE((rows.rid2 >= 0) == (cols.rid2 >= 0) && rows.rid2 == cols.rid2 &&
                 rows.variant == cols.variant && rows.r2max == cols.r2max,
             FD_ERR_INVALID_ARG, "internal: pack layouts do not match");
  ProfScope prof(kind, stream);
  go(rows, cols);
  if (rows.rid2 >= 0) go(full_offset_view(rows), full_offset_view(cols));
}

void launch_product_hx(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                       const float* vp, const float* cs, bool diag, const float* sl, float* Y,
                       int64_t ldy, int b, float* part, hipStream_t stream) {
  dual_dispatch(rows, cols, FD_KERNEL_PRODUCT, stream, [&](const PointPack& r, const PointPack& c) {
    check_hx(p, r, c);
    switch (r.rid) {
      case 0: return product_hx_ncb<0>(p, r, c, vp, cs, diag, sl, Y, ldy, b, part, stream);
      case 1: return product_hx_ncb<1>(p, r, c, vp, cs, diag, sl, Y, ldy, b, part, stream);
      case 2: return product_hx_ncb<2>(p, r, c, vp, cs, diag, sl, Y, ldy, b, part, stream);
      case 3: return product_hx_ncb<3>(p, r, c, vp, cs, diag, sl, Y, ldy, b, part, stream);
      case 4: return product_hx_ncb<4>(p, r, c, vp, cs, diag, sl, Y, ldy, b, part, stream);
      case 5: return product_hx_ncb<5>(p, r, c, vp, cs, diag, sl, Y, ldy, b, part, stream);
      case 6: return product_hx_ncb<6>(p, r, c, vp, cs, diag, sl, Y, ldy, b, part, stream);
    }
  });
}

void launch_rowsum_sym_hx(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                          const float* wp, float* part, unsigned long long* colfix,
                          double fix_scale, const SymSquares& sq, hipStream_t stream) {
  FD_REQUIRE(rows.rid >= 0 && rows.rid < HX_RECIPES && rows.rid == cols.rid && rows.row_side &&
                 !cols.row_side && rows.n == cols.n,
             FD_ERR_INVALID_ARG, "internal: symmetric row sums need one point set");
  FD_REQUIRE((p.nib == 4 || p.nib == 8) && p.nrt * 4 * p.nib * TILE == rows.npad &&
                 p.njb == ceil_div(cols.n, TILE),
             FD_ERR_INVALID_ARG, "internal: symmetric row-sum plan");
  dual_dispatch(rows, cols, FD_KERNEL_ROWSUM, stream, [&](const PointPack& r, const PointPack& c) {
    const HxRecipe& R = HX_TABLE[r.rid];
    check_span(r.xp, size_t(r.npad / TILE) * R.nb * 64 * 4, "split row pack");
    check_span(c.xp, size_t(round_up(p.njb, 2)) * R.nc * 64 * 4, "split column pack");
    switch (r.rid) {
      case 0: return rowsum_sym_hx_u<0>(p, r, c, wp, part, colfix, fix_scale, sq, stream);
      case 1: return rowsum_sym_hx_u<1>(p, r, c, wp, part, colfix, fix_scale, sq, stream);
      case 2: return rowsum_sym_hx_u<2>(p, r, c, wp, part, colfix, fix_scale, sq, stream);
      case 3: return rowsum_sym_hx_u<3>(p, r, c, wp, part, colfix, fix_scale, sq, stream);
      case 4: return rowsum_sym_hx_u<4>(p, r, c, wp, part, colfix, fix_scale, sq, stream);
      case 5: return rowsum_sym_hx_u<5>(p, r, c, wp, part, colfix, fix_scale, sq, stream);
      case 6: return rowsum_sym_hx_u<6>(p, r, c, wp, part, colfix, fix_scale, sq, stream);
    }
  });
}

void launch_rowsum_hx(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                      const float* wp, bool diag, float* out, float* part, hipStream_t stream) {
  FD_REQUIRE(p.nib == 4 || p.nib == 8, FD_ERR_INVALID_ARG, "internal: row-sum plan");
  dual_dispatch(rows, cols, FD_KERNEL_ROWSUM, stream, [&](const PointPack& r, const PointPack& c) {
    check_hx(p, r, c);
    switch (r.rid) {
      case 0: return rowsum_hx_u<0>(p, r, c, wp, diag, out, part, stream);
      case 1: return rowsum_hx_u<1>(p, r, c, wp, diag, out, part, stream);
      case 2: return rowsum_hx_u<2>(p, r, c, wp, diag, out, part, stream);
      case 3: return rowsum_hx_u<3>(p, r, c, wp, diag, out, part, stream);
      case 4: return rowsum_hx_u<4>(p, r, c, wp, diag, out, part, stream);
      case 5: return rowsum_hx_u<5>(p, r, c, wp, diag, out, part, stream);
      case 6: return rowsum_hx_u<6>(p, r, c, wp, diag, out, part, stream);
    }
  });
}

}  // namespace fd
