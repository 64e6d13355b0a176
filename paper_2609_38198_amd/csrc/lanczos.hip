// Block Lanczos eigensolver and (n, beta) continuation.
#include "fd_solver.hpp"

namespace fd {

void carve_solver(Arena& a, int64_t N, int64_t D, int b, int k, const fd_lanczos_opts& o,
                  bool continuation) {
  (void)a; (void)N; (void)D; (void)b; (void)k; (void)o; (void)continuation;
}

}  // namespace fd

extern "C" {

fd_status fd_block_lanczos(const void*, fd_dtype, int64_t, int64_t, int64_t, float, float, int64_t,
                           int64_t, const float*, int64_t, int64_t, int32_t,
                           const fd_lanczos_opts*, double*, float*, float*, double*,
                           fd_lanczos_info*, void*, size_t, void*) {
  fd::set_error("block Lanczos not built yet");
  return FD_ERR_UNSUPPORTED;
}

fd_status fd_continuation(const void*, fd_dtype, int64_t, int64_t, int64_t, float, const int64_t*,
                          const float*, int64_t, int64_t, int64_t, const float*, int64_t, int64_t,
                          const fd_lanczos_opts*, double*, float*, float*, fd_lanczos_info*,
                          int32_t, int64_t*, void*, size_t, void*) {
  fd::set_error("continuation not built yet");
  return FD_ERR_UNSUPPORTED;
}

}  // extern "C"
