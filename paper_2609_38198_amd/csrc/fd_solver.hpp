// Composite operations shared by the entry points and the eigensolver.
#pragma once

#include "fd_internal.hpp"

namespace fd {

// Workspace of one fused product: packed rows / columns, packed V, partials.
struct ProductWs {
  PointPack rows, cols;
  FSpan vp, vscale, part;
  FSpan tmp;  // one float per row: the single-column product's row sums
  int* flag = nullptr;  // set when a point set holds a non-finite value
  CentreWs centre;      // common centre of the row and column sets
  KVPlan plan;
};

// Workspace of the two normalisation passes.
struct DegreeWs {
  PointPack rows, cols;
  FSpan wp, part;
  float* q = nullptr;
  float* t = nullptr;
  float* w = nullptr;
  unsigned long long* colfix = nullptr;  // npad words: column sums of the symmetric row sums
  FSpan sq_part;                          // squared-kernel row partials (dyadic levels)
  unsigned long long* sq_colfix = nullptr;
  int* flag = nullptr;  // set when X holds a non-finite value
  CentreWs centre;      // centre of X
  KVPlan plan;
};

void check_points(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx, const char* what);
void check_workspace(const void* ws, size_t ws_bytes, size_t need);

ProductWs carve_product(Arena& a, int64_t Nr, int64_t Nc, int64_t D, int b);
// Y = diag(sl) K diag(sr) V with the packs already filled.
void product_apply(ProductWs& w, const float* sl, const float* sr, const float* V, int64_t ldv,
                   int b, float* Y, int64_t ldy, bool diag, hipStream_t stream);

DegreeWs carve_degree(Arena& a, int64_t N, int64_t D);
// q, d, s (any may be NULL) and s_off; `pack` = fill the point packs first.
void degree_run(DegreeWs& w, const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                double beta, double alpha, float* q, float* d, float* s, double* s_off,
                bool pack, hipStream_t stream);

// carve_degree plus the squared-kernel buffers of the dyadic ladder.
DegreeWs carve_degree_dyadic(Arena& a, int64_t N, int64_t D);
// Levels l = 0 .. nb - 1 at beta0 2^l: q, d, s at offset l N (each may be NULL),
// s_off[l] (or NULL).
void degree_run_dyadic(DegreeWs& w, const void* X, fd_dtype xt, int64_t N, int64_t D,
                       int64_t ldx, double beta0, int nb, double alpha, float* q, float* d,
                       float* s, double* s_off, hipStream_t stream);

// Non-finite inputs.  scan: clear *flag, then set it if any of the N x D
// values of X is NaN or infinite.  poison: when *flag is set, fill rows x cols
// floats of v (leading dimension ld) with NaN.  Both asynchronous.
void launch_scan_nonfinite(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx,
                           int* flag, bool clear, hipStream_t stream);
void launch_poison(const int* flag, float* v, int64_t rows, int64_t cols, int64_t ld,
                   hipStream_t stream);
void launch_poison(const int* flag, double* v, int64_t n, hipStream_t stream);
// Synchronous check for the eigensolver entry points: FD_ERR_INVALID_ARG when
// X holds a non-finite value.
void require_finite(const void* X, fd_dtype xt, int64_t N, int64_t D, int64_t ldx, int* flag,
                    hipStream_t stream);

// Row slots of a partial-sum buffer large enough for every plan with at most
// npad rows and nc columns (see plan_product).
size_t part_rows_bound(int64_t npad, int64_t nc);
// Views of workspace carved for a larger problem, for n <= the carved size.
PointPack pack_view(const PointPack& big, int64_t n, int64_t pad);
DegreeWs degree_view(const DegreeWs& big, int64_t n);
ProductWs product_view(const ProductWs& big, const PointPack& rows, const PointPack& cols,
                       int width);

// Eigensolver workspace (sizes only when a.measuring).
void carve_solver(Arena& a, int64_t N, int64_t D, int b, int k, const fd_lanczos_opts& o);
void carve_continuation_ws(Arena& a, int64_t nmax, int64_t nsteps, int64_t D, int b, int k,
                           const fd_lanczos_opts& o);
void carve_flow_ws(Arena& a, int64_t N, int64_t D, int b, int k, const fd_lanczos_opts& o);

}  // namespace fd
