// Composite operations shared by the entry points and the eigensolver.
#pragma once

#include "fd_internal.hpp"

namespace fd {

// Workspace of one fused product: packed rows / columns, packed V, partials.
struct ProductWs {
  PointPack rows, cols;
  FSpan vp, part;
  KVPlan plan;
};

// Workspace of the two normalisation passes.
struct DegreeWs {
  PointPack rows, cols;
  FSpan wp, part;
  float* q = nullptr;
  float* t = nullptr;
  float* w = nullptr;
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

// Eigensolver workspace (sizes only when a.measuring).
void carve_solver(Arena& a, int64_t N, int64_t D, int b, int k, const fd_lanczos_opts& o,
                  bool continuation);

}  // namespace fd
