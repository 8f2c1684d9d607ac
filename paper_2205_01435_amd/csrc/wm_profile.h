// Opt-in per-kernel timing of libwm launches with HIP events (a measurement
// aid behind wm_profile_enable / wm_profile_read).
#pragma once

#include <hip/hip_runtime.h>

namespace wm {

// Brackets one kernel launch: records a start event on construction and a
// stop event on destruction, on the launch stream, when profiling is enabled
// for a prefix of `name`.
class KTimer {
 public:
  KTimer(const char* name, hipStream_t s);
  ~KTimer();
  KTimer(const KTimer&) = delete;
  KTimer& operator=(const KTimer&) = delete;

 private:
  const char* name_;
  hipStream_t s_;
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

}  // namespace wm
