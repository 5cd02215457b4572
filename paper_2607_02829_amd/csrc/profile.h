// Optional per-launch timing with HIP events (off unless sr_profile_start is called).
// A scope binds a start event to the first kernel it launches and a stop event to the last
// (the launch hook of common.h), so its interval is that of its kernels' own execution;
// a scope that launches nothing records both events where it ends.  sr_profile_stop sums
// elapsed times per name.
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
  hipEvent_t outer_start_ = nullptr, outer_stop_ = nullptr;   // the enclosing binding, restored at the end
  unsigned long long launches0_ = 0;
};

}  // namespace sr
