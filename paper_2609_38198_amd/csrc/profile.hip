// Optional per-kernel timing with HIP events recorded on the launch stream.
#include <mutex>
#include <utility>
#include <vector>

#include "fd_internal.hpp"
#include "fd_profile.hpp"

namespace fd {

namespace {
struct Pool {
  std::mutex m;
  bool on = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev[FD_KERNEL_KINDS];
  size_t used[FD_KERNEL_KINDS] = {};
};
Pool& pool() {
  static Pool p;
  return p;
}
constexpr size_t MAX_EVENTS = 1 << 16;
}  // namespace

ProfScope::ProfScope(int kind, hipStream_t s) : stream_(s) {
  Pool& p = pool();
  std::lock_guard<std::mutex> g(p.m);
  if (!p.on || kind < 0 || kind >= FD_KERNEL_KINDS) return;
  auto& v = p.ev[kind];
  size_t& u = p.used[kind];
  if (u >= MAX_EVENTS) return;
  if (u == v.size()) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return;
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return;
    }
    v.emplace_back(a, b);
  }
  start_ = v[u].first;
  stop_ = v[u].second;
  ++u;
  (void)hipEventRecord(start_, stream_);
}

ProfScope::~ProfScope() {
  if (stop_ != nullptr) (void)hipEventRecord(stop_, stream_);
}

}  // namespace fd

extern "C" {

void fd_profile_enable(int32_t on) {
  fd::Pool& p = fd::pool();
  std::lock_guard<std::mutex> g(p.m);
  p.on = on != 0;
}

fd_status fd_profile_read(fd_kernel_kind kind, double* total_ms, int64_t* launches) {
  fd::Pool& p = fd::pool();
  std::lock_guard<std::mutex> g(p.m);
  if (int(kind) < 0 || int(kind) >= fd::FD_KERNEL_KINDS || total_ms == nullptr ||
      launches == nullptr) {
    fd::set_error("fd_profile_read: bad argument");
    return FD_ERR_INVALID_ARG;
  }
  double sum = 0.0;
  const size_t u = p.used[kind];
  for (size_t i = 0; i < u; ++i) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(p.ev[kind][i].second);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.ev[kind][i].first, p.ev[kind][i].second);
    if (e != hipSuccess) {
      fd::set_error(std::string("fd_profile_read: ") + hipGetErrorString(e));
      return FD_ERR_HIP;
    }
    sum += ms;
  }
  *total_ms = sum;
  *launches = int64_t(u);
  p.used[kind] = 0;
  return FD_OK;
}

}  // extern "C"
