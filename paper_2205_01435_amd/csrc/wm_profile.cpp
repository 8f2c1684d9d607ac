// Per-kernel timing for measurement runs (wm_profile_* entry points): event
// pairs stamped by the kernel dispatches (see launch() in wm_profile.h).
#include "wm_profile.h"

#include <stdint.h>

#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/wm.h"

namespace wm {
namespace {

struct Rec {
  std::string name;
  hipEvent_t a, b;
};

std::mutex g_mu;
bool g_on = false;
std::string g_prefix;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

bool starts_with(const std::string& s, const char* p) {
  return std::strncmp(s.c_str(), p, std::strlen(p)) == 0;
}

}  // namespace

KTimer::KTimer(const char* name) : name_(name) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on || std::strncmp(name, g_prefix.c_str(), g_prefix.size()) != 0) return;
  a_ = take_event();
  b_ = take_event();
  if (a_ && b_) return;
  if (a_) g_pool.push_back(a_);
  if (b_) g_pool.push_back(b_);
  a_ = b_ = nullptr;
}

void KTimer::commit() {
  if (!a_ || !b_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  g_recs.push_back(Rec{name_, a_, b_});
  a_ = b_ = nullptr;
}

KTimer::~KTimer() {
  if (!a_ && !b_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (a_) g_pool.push_back(a_);
  if (b_) g_pool.push_back(b_);
}

}  // namespace wm

extern "C" {

wm_status wm_profile_enable(const char* prefix) {
  std::lock_guard<std::mutex> lk(wm::g_mu);
  wm::g_on = prefix != nullptr;
  wm::g_prefix = prefix ? prefix : "";
  return WM_OK;
}

wm_status wm_profile_read(const char* prefix, double* total_ms, int64_t* launches) {
  if (!total_ms || !launches) return WM_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(wm::g_mu);
  double tot = 0.0;
  int64_t n = 0;
  for (const wm::Rec& r : wm::g_recs) {
    if (prefix && !wm::starts_with(r.name, prefix)) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) return WM_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return WM_ERR_HIP;
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return WM_OK;
}

wm_status wm_profile_reset(void) {
  std::lock_guard<std::mutex> lk(wm::g_mu);
  for (const wm::Rec& r : wm::g_recs) {
    (void)hipEventSynchronize(r.b);
    wm::g_pool.push_back(r.a);
    wm::g_pool.push_back(r.b);
  }
  wm::g_recs.clear();
  return WM_OK;
}

}  // extern "C"
