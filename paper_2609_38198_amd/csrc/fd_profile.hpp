// RAII bracket of one kernel launch with HIP events (active only when
// fd_profile_enable(1) was called).
#pragma once

#include <hip/hip_runtime.h>

#include "flashdiff.h"

namespace fd {

constexpr int FD_KERNEL_KINDS = 2;

class ProfScope {
 public:
  ProfScope(int kind, hipStream_t s);
  ~ProfScope();
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
  hipEvent_t stop_ = nullptr;
};

}  // namespace fd
