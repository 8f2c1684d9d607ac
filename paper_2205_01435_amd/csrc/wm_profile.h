// Kernel launches of libwm, with opt-in per-kernel timing (wm_profile_enable
// / wm_profile_read): when timing is enabled for a prefix of a launch's name,
// the launch carries a start/stop event pair that the dispatch itself stamps
// (hipExtLaunchKernel), so the recorded interval is the kernel's own run.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <tuple>
#include <utility>

namespace wm {

class KTimer {
 public:
  explicit KTimer(const char* name);  // takes an event pair if timing is on for name
  ~KTimer();                          // returns unused events to the pool
  KTimer(const KTimer&) = delete;
  KTimer& operator=(const KTimer&) = delete;
  hipEvent_t start() const { return a_; }
  hipEvent_t stop() const { return b_; }
  void commit();  // the launch went out: keep the pair for wm_profile_read

 private:
  const char* name_;
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

namespace detail {
template <typename Tup, size_t... I>
void arg_ptrs(Tup& t, void** p, std::index_sequence<I...>) {
  ((p[I] = static_cast<void*>(&std::get<I>(t))), ...);
}
}  // namespace detail

// Phase timing of the persistent kernels (wm_profile_phases): while it is
// on, a device buffer of at least `words` zeroed 64-bit words (allocated on
// first use, grown as needed) for the stamps of the next launch; null while
// it is off.
unsigned long long* phase_buffer(size_t words, hipStream_t s);
// Layout of the launch that takes the stamps: `groups` work-groups of `nst`
// stamps each, T steps, the NLL recurrence or the rollout.
void phase_layout(int groups, int nst, int T, bool nll);

// Launches kernel<<<grid, block, shm, s>>>(args...) and returns the launch
// status.
template <typename... P, typename... A>
hipError_t launch(const char* name, void (*kernel)(P...), dim3 grid, dim3 block, size_t shm,
                  hipStream_t s, A... args) {
  static_assert(sizeof...(P) == sizeof...(A), "argument count");
  std::tuple<P...> tup{static_cast<P>(args)...};
  void* ptrs[sizeof...(P) > 0 ? sizeof...(P) : 1];
  detail::arg_ptrs(tup, ptrs, std::index_sequence_for<P...>{});
  KTimer kt(name);
  const hipError_t e = hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs,
                                          shm, s, kt.start(), kt.stop(), 0);
  if (e == hipSuccess) kt.commit();
  return e;
}

}  // namespace wm
