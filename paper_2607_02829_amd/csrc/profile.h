// Optional per-launch timing with HIP events (off unless sr_profile_start is called).
// A scope records an event before and after the launches it wraps, on the stream they
// are launched on; sr_profile_stop sums elapsed times per name.
#pragma once
#include <hip/hip_runtime.h>

namespace sr {

bool profiling();
// Profiling every launch group (no name filter): launches that normally overlap on a
// second stream are issued on the caller's stream instead, so each group's time is its own.
bool profiling_all();

class ProfScope {
 public:
  ProfScope(const char* name, double flops, double bytes, hipStream_t st);
  ~ProfScope();
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  int slot_ = -1;
  hipStream_t st_;
};

}  // namespace sr
