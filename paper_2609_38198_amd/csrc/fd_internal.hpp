// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "flashdiff.h"

namespace fd {

// ---------------------------------------------------------------- errors
void set_error(const std::string& msg);
const char* get_error();

struct Error {
  fd_status status;
  std::string msg;
};

#define FD_HIP_CHECK(expr)                                                               \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      throw ::fd::Error{FD_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)}; \
  } while (0)

#define FD_LAUNCH_CHECK() FD_HIP_CHECK(hipGetLastError())

#define FD_REQUIRE(cond, status, msg)                 \
  do {                                                \
    if (!(cond)) throw ::fd::Error{(status), (msg)}; \
  } while (0)

// ---------------------------------------------------------------- workspace
// A carved region of float32 elements.
struct FSpan {
  float* p = nullptr;
  size_t n = 0;
};

inline void check_span(const FSpan& s, size_t need, const char* what) {
  if (s.p == nullptr || s.n < need)
    throw Error{FD_ERR_WORKSPACE, std::string("internal: region '") + what +
                                      "' smaller than the extent its kernel touches"};
}

// Bump allocator over the caller's workspace (never allocates device memory).
struct Arena {
  char* base = nullptr;
  size_t cap = 0;
  size_t used = 0;
  bool measuring = false;  // when true only counts bytes
  template <class T>
  T* take(size_t count) {
    size_t bytes = (count * sizeof(T) + 255) & ~size_t(255);
    size_t off = used;
    used += bytes;
    if (measuring) return nullptr;
    if (used > cap) throw Error{FD_ERR_WORKSPACE, "workspace too small"};
    return reinterpret_cast<T*>(base + off);
  }
  FSpan fspan(size_t count) { return FSpan{take<float>(count), count}; }
};

// ---------------------------------------------------------------- geometry
constexpr int TILE = 16;          // points per MFMA tile
constexpr int WG_THREADS = 256;   // four wave64 per workgroup
constexpr int ROW_PAD = 512;      // row packs: whole workgroups of 4 waves x 8 row tiles
constexpr int COL_PAD = 32;       // column packs: whole pairs of 16-point tiles
// Longest column range one workgroup of a product or row-sum plan streams
// (tiles of 16 points); longer ranges are split.  The workgroups that run
// together on an XCD start a split together and drift apart; over 4,096
// tiles (a few tens of MB of column operands) their working set stays
// cache-resident, over 32,768 it did not always (the bfloat16 product at
// N = 2^21, b = 64 then ran 1.5 to 2.2 s against 1.43 s).
constexpr int64_t SPLIT_SPAN_TILES = 4096;

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline int64_t ceil_div(int64_t x, int64_t m) { return (x + m - 1) / m; }

// Padded contraction width used for a feature dimension D (multiple of 4).
int padded_dim(int64_t D);
// Supported feature dimensions and block widths.
constexpr int MAX_D = 64;
constexpr int MAX_B = 64;

// Packed operands of one point set, produced by launch_pack_points.
// float32 X: xp holds the split float16 exponent chunks ([tiles][chunks][64]
//   uint4; chunk layout by recipe rid, row or column side).
// bfloat16 X: xp holds [tiles][dc][64] uint4 of raw bfloat16 features,
//   ap [tiles][64][4] the column offsets -||x_j||^2/2 in accumulator order,
//   ar [npad] the row offsets.
struct PointPack {
  FSpan xp, ap, ar;
  int64_t n = 0;      // real points
  int64_t npad = 0;   // padded points
  int dp = 0;         // padded feature width the region was sized for
  bool bf16 = false;  // filled from bfloat16 X
  int dc = 0;         // bfloat16: 32-feature chunks
  int rid = -1;       // float32: split-exponent recipe
  bool row_side = false;
  double beta = 0.0;  // bandwidth the pack was made for
  // float32 packs of a D whose short layout drops the third offset piece
  // (13 < D <= 30, 32 < D <= 62): the layout with all three pieces too (xp2,
  // recipe rid2), and the device word the kernels choose between them by
  // (max ||x - mu||^2 as float64 bits); variant 1 / 2 = this pack is the
  // short / the full-offset one, 0 = no choice.
  FSpan xp2;
  int rid2 = -1;
  const unsigned long long* r2max = nullptr;
  int variant = 0;
};

// Centring of a float32 point set (the kernel is translation invariant, and
// the Gram-form exponent is most accurate around the mean): column means mu
// (float64) and the largest squared distance of a point from them.
struct CentreWs {
  double* part = nullptr;             // nblk x D column partial sums
  double* mu = nullptr;               // D
  unsigned long long* r2max = nullptr;  // float64 bits of max ||x - mu||^2
  int nblk = 0;
};
CentreWs carve_centre(Arena& a, int64_t n);
// mu of X[0:n] and r2max over it (float32 X; a no-op for bfloat16).
void launch_centre(const void* X, fd_dtype xt, int64_t n, int64_t D, int64_t ldx,
                   const CentreWs& c, hipStream_t stream);
// r2max also over X2[0:n2], centred on the same mu.
void launch_radius_more(const void* X2, fd_dtype xt, int64_t n2, int64_t D, int64_t ldx,
                        const CentreWs& c, hipStream_t stream);

// Exponent budget of the short split layouts: above beta log2(e) max ||x - mu||^2
// = 64 the kernels take the layout that keeps all three offset pieces (the
// dropped third piece is a coherent row / column scale error of up to
// 2^-22 ln 2 times that, 3.7e-6 relative at 64, against measured K V errors of
// 2.8e-6 at 50 and 5.4e-6 at 100 on the molecule-like set).
constexpr double EXP_BUDGET = 64.0;

// Exponent range of the float32 path: the row and column offsets
// -beta log2(e) ||x - mu||^2 (+15 on the row side) enter the contraction as
// float16 pieces, which hold magnitudes up to 65504.  Above
// beta log2(e) max ||x - mu||^2 = HX_EXP_RANGE the exponent cannot be formed:
// the asynchronous entry points fill their outputs with NaN, the synchronous
// ones refuse (FD_ERR_UNSUPPORTED) and the flow stops before such a probe.
// (bfloat16 X forms its exponent in float32 and has no such limit.)
constexpr double HX_EXP_RANGE = 65504.0 - 16.0;
// The coordinates enter as float16 pieces of s (x - mu) (column side) and
// 2 beta log2(e) (x - mu) / s (row side): both must stay within 65504 too.
// The balanced s keeps them below 512 inside the offset range; only its clamp
// at the float32 extremes of beta (below about 1e-39) could break that.
constexpr double HX_PIECE_MAX = 65504.0;
// s of the float32 packs for bandwidth beta (a power of two).
double hx_coord_scale(double beta);
// Whether bandwidth beta is inside the exponent range (offsets and
// coordinate pieces) for points of squared centred radius r2max (always for
// bfloat16 X).
bool exponent_in_range(fd_dtype xt, double beta, double r2max);
// r2max of a centring (host copy; synchronises the stream; 0 for bfloat16).
double exponent_radius(fd_dtype xt, const CentreWs& c, hipStream_t stream);
// Synchronous check: FD_ERR_UNSUPPORTED when beta is outside the range.
void require_exponent_range(fd_dtype xt, const CentreWs& c, double beta, hipStream_t stream);
// Asynchronous check: sets bit 2 of *flag (the non-finite-input flag, whose
// poison fills the outputs with NaN) when beta is outside the range.
void launch_range_check(fd_dtype xt, const CentreWs& c, double beta, int* flag,
                        hipStream_t stream);

// Floats per point of a pack region (large enough for either pack kind).
int pack_floats_per_point(int64_t D);

// Plan of one fused product / degree launch.
struct KVPlan {
  int dp = 0, ncb = 0, nib = 0;
  int64_t njb = 0;        // column tiles of 16
  int64_t nrt = 0;        // row tiles of 64*nib
  int nsplit = 1;         // column splits
  int64_t jb_per_split = 0;
};

// Tiling of a fused product (rows per wave tuned by shape) and of a row sum.
KVPlan plan_tiles(int64_t Nr, int64_t Nc, int dp, int b, int nib);
int product_nib(int dp, int ncb);
KVPlan plan_product(int64_t Nr, int64_t Nc, int dp, int b);
KVPlan plan_rowsum(int64_t Nr, int64_t Nc, int dp);

// Workspace carving helpers (size when arena.measuring).
PointPack carve_pack(Arena& a, int64_t n, int dp, int64_t pad);

// Launchers (enqueue on stream; throw Error on failure).
void launch_pack_points(const void* X, fd_dtype xt, int64_t n, int64_t D, int64_t ldx,
                        double beta, bool row_side, PointPack& out, const CentreWs* centre,
                        hipStream_t stream);
void launch_pack_w(const float* w, int64_t n, int64_t npad, FSpan wp, hipStream_t stream);
// Weight pack of sr * v for one column v (row stride ldv; sr may be NULL).
void launch_pack_wv(const float* v, int64_t ldv, const float* sr, int64_t n, int64_t npad,
                    FSpan wp, hipStream_t stream);
// Y[i * ldy] = sl[i] * t[i] (sl NULL: t[i]).
void launch_scale_rows(const float* t, const float* sl, int64_t n, float* Y, int64_t ldy,
                       hipStream_t stream);
// Pack sr * V for the product that matches the row pack's kind.
void launch_pack_v_for(const PointPack& rows, const float* V, int64_t n, int64_t b, int64_t ldv,
                       const float* sr, int ncb, int64_t npad, FSpan vp, FSpan vscale,
                       hipStream_t stream);
// Split float16 pack of sr * V with per-column power-of-two scales (vscale:
// 64 max-abs bit patterns followed by 64 inverse scales).
void launch_pack_v_split(const float* V, int64_t n, int64_t b, int64_t ldv, const float* sr,
                         int ncb, int64_t npad, FSpan vp, FSpan vscale, hipStream_t stream);
// Y = diag(sl) K diag(sr) V from packed operands (V packed with sr applied).
void launch_product(const KVPlan& p, const PointPack& rows, const PointPack& cols, FSpan vp,
                    FSpan vscale, bool diag, const float* sl, float* Y, int64_t ldy, int b,
                    FSpan part, hipStream_t stream);
// out = K w (wp.p == NULL: w = 1).  With colfix (npad 64-bit words of
// scratch) and rows and columns the same float32 point set, the symmetric
// kernel is used (weights must lie in [0, 1]).
void launch_rowsum(const KVPlan& p, const PointPack& rows, const PointPack& cols, FSpan wp,
                   bool diag, float* out, FSpan part, hipStream_t stream,
                   unsigned long long* colfix = nullptr);
KVPlan plan_rowsum_sym(int64_t N, int64_t npad, int dp, int nib);
// The symmetric path piece by piece (the two normalisation passes fuse their
// epilogues into its reduction): whether it applies, one pass of the kernel
// (row partials in part, fixed-point column sums added into colfix, which is
// zeroed first if asked), and the fused reductions.  Each reduction leaves
// colfix zeroed.  launch_degree_reduce_q: q, and w = q^-alpha into the weight
// pack (the column pack's extent) when wp.p is set; launch_degree_reduce_ds: d = w t and s = w d^-1/2
// (either may be NULL).
struct SymPass {
  int nsplit = 0;
  double inv_fix = 0.0;
};
// Second output of a weighted symmetric pass: the unit-weight row sums (per
// split, part) and fixed-point column sums (colfix) of the squared kernel.
struct SymSquares {
  float* part = nullptr;
  unsigned long long* colfix = nullptr;
  double fix_scale = 0.0;
};
bool rowsum_sym_applies(const PointPack& rows, const PointPack& cols, bool diag,
                        const unsigned long long* colfix);
// sq_part / sq_colfix (weighted passes only): also the squared-kernel sums, whose
// reduction uses the returned inv_fix as well.
SymPass launch_rowsum_sym_pass(const KVPlan& p, const PointPack& rows, const PointPack& cols,
                               FSpan wp, FSpan part, unsigned long long* colfix, bool zero_colfix,
                               hipStream_t stream, FSpan sq_part = FSpan{},
                               unsigned long long* sq_colfix = nullptr);
void launch_degree_reduce_q(const SymPass& sp, const PointPack& rows, const PointPack& cols,
                            FSpan part, unsigned long long* colfix, float* q, double alpha,
                            FSpan wp, hipStream_t stream);
void launch_degree_reduce_ds(const SymPass& sp, const PointPack& rows, FSpan part,
                             unsigned long long* colfix, const float* q, double alpha, float* d,
                             float* s, hipStream_t stream);
// launch_degree_reduce_ds plus the squared-kernel sums of the same pass: the
// next dyadic level's q_next = K(2 beta) 1 and its w = q_next^-alpha into the
// weight pack wp (the column pack's extent); leaves both colfix arrays zeroed.
void launch_degree_reduce_dsq(const SymPass& sp, const PointPack& rows, const PointPack& cols,
                              FSpan part, unsigned long long* colfix, const float* q,
                              double alpha, float* d, float* s, FSpan sq_part,
                              unsigned long long* sq_colfix, float* q_next, FSpan wp,
                              hipStream_t stream);
void launch_zero_u64(unsigned long long* p, int64_t n, hipStream_t stream);
// Row tiles per wave of the symmetric row sums, and the fewest column splits
// of their large-problem plans.
constexpr int SYM_NIB = 8;
constexpr int64_t SYM_MIN_SPLITS = 16;
// Row slots of the partial sums of a symmetric row-sum plan with npad rows.
size_t sym_part_rows(int64_t npad, int nib);
void launch_degree_finish(const float* q, const float* t, int64_t n, double alpha, float* d,
                          float* s, hipStream_t stream);
void launch_pow_neg(const float* q, int64_t n, double alpha, float* w, hipStream_t stream);
void launch_sum_minus_n(const float* q, int64_t n, double* out, hipStream_t stream);

}  // namespace fd
