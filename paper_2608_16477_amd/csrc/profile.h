// Per-kernel timing: HIP event pairs around launches of enabled classes.
#pragma once

#include <hip/hip_runtime.h>

#include "pallas.h"

namespace pallas {

bool profile_on(int cls);
void profile_record(int cls, hipEvent_t begin, hipEvent_t end);
hipEvent_t profile_event();
// Device counters [cycles, wall ticks, workgroups] for clock sampling inside
// the launches of `cls`, or null when the class is not being timed.
unsigned long long* profile_clock_slot(int cls);

// Brackets the launches issued during its lifetime on `s`.
class ProfScope {
 public:
  ProfScope(int cls, hipStream_t s) : cls_(cls), s_(s) {
    if (profile_on(cls)) {
      begin_ = profile_event();
      if (begin_) (void)hipEventRecord(begin_, s_);
    }
  }
  ~ProfScope() {
    if (!begin_) return;
    hipEvent_t end = profile_event();
    if (end && hipEventRecord(end, s_) == hipSuccess) profile_record(cls_, begin_, end);
  }
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  int cls_;
  hipStream_t s_;
  hipEvent_t begin_ = nullptr;
};

}  // namespace pallas
