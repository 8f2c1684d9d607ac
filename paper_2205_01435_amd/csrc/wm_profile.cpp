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

// ---------------------------------------------------------------------------
// Phase stamps of the persistent kernels
// ---------------------------------------------------------------------------
namespace {
std::mutex g_pmu;
bool g_phases = false;
unsigned long long* g_pbuf = nullptr;
size_t g_pwords = 0;
int g_pgroups = 0, g_pnst = 0, g_pT = 0;
bool g_pnll = false;
}  // namespace

unsigned long long* phase_buffer(size_t words, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_pmu);
  if (!g_phases) return nullptr;
  if (words > g_pwords) {
    if (g_pbuf) (void)hipFree(g_pbuf);
    g_pbuf = nullptr;
    g_pwords = 0;
    if (hipMalloc(&g_pbuf, words * 8) != hipSuccess) {
      g_pbuf = nullptr;
      return nullptr;
    }
    g_pwords = words;
  }
  if (hipMemsetAsync(g_pbuf, 0, words * 8, s) != hipSuccess) return nullptr;
  return g_pbuf;
}

void phase_layout(int groups, int nst, int T, bool nll) {
  std::lock_guard<std::mutex> lk(g_pmu);
  g_pgroups = groups;
  g_pnst = nst;
  g_pT = T;
  g_pnll = nll;
}

}  // namespace wm

namespace {

// Per-step phase durations (us) from the stamps of one launch; see
// wm_profile_phases_read for the slots of `out`.
void phase_summary(const std::vector<unsigned long long>& st, int groups, int nst, int T, bool nll,
                   double tick_us, double* out) {
  constexpr int kX = 8;  // work-groups g with g % 8 == x form XCD group x
  const int per = groups / kX;
  auto at = [&](int g, int i) { return st[(size_t)g * nst + i]; };
  auto arrive = [&](int g, int b) { return at(g, 2 * b - 1); };
  auto release = [&](int g, int b) { return at(g, 2 * b); };
  double acc[13] = {0};
  int nx = 0;
  for (int x = 0; x < kX; ++x) {
    bool whole = true;
    for (int k = 0; k < per && whole; ++k)
      for (int i = 0; i < nst; ++i)
        if (at(x + kX * k, i) == 0) { whole = false; break; }
    if (!whole) continue;  // a group without rows (or stopped early)
    ++nx;
    // phase ending at barrier b (or at the end, b = 0): max and mean over
    // the group of (arrival - release of the previous barrier pb)
    auto work = [&](int pb, int b, double& mx, double& mean) {
      double m = 0, sum = 0;
      for (int k = 0; k < per; ++k) {
        const int g = x + kX * k;
        const double d = (double)((b ? arrive(g, b) : at(g, nst - 1)) - (pb ? release(g, pb) : at(g, 0)));
        m = d > m ? d : m;
        sum += d;
      }
      mx += m * tick_us;
      mean += sum / per * tick_us;
    };
    // the barrier's own latency: first release after the last arrival
    auto latency = [&](int b) {
      unsigned long long last = 0, first = ~0ull;
      for (int k = 0; k < per; ++k) {
        const int g = x + kX * k;
        last = arrive(g, b) > last ? arrive(g, b) : last;
        first = release(g, b) < first ? release(g, b) : first;
      }
      return (double)(first - last) * tick_us;
    };
    auto first_release = [&](int b) {
      unsigned long long f = ~0ull;
      for (int k = 0; k < per; ++k) f = release(x + kX * k, b) < f ? release(x + kX * k, b) : f;
      return f;
    };
    auto last_end = [&]() {
      unsigned long long l = 0;
      for (int k = 0; k < per; ++k) l = at(x + kX * k, nst - 1) > l ? at(x + kX * k, nst - 1) : l;
      return l;
    };
    double dummy = 0, pro = 0, epi = 0;
    if (nll) {
      // barrier 1 ends the set-up; barrier 1 + t + 1 follows step t < T - 1
      for (int t = 0; t < T; ++t) {
        const int b = t + 1 < T ? t + 2 : 0;
        work(t + 1, b, acc[4], acc[9]);
        if (b) acc[5] += latency(b);
      }
      acc[1] += (double)(last_end() - first_release(1)) * tick_us / T;
      work(0, 1, pro, dummy);
    } else {
      // barriers 1, 2 end the set-up; 3 + 2t and 4 + 2t follow gates(t)
      // (which makes the step's controller decisions) and mdn(t)
      for (int t = 0; t < T; ++t) {
        const int b = 3 + 2 * t;
        work(b - 1, b, acc[4], acc[9]);
        acc[5] += latency(b);
        work(b, b + 1, acc[6], acc[10]);
        acc[7] += latency(b + 1);
      }
      acc[1] += (double)(first_release(2 + 2 * T) - first_release(2)) * tick_us / T;
      work(0, 2, pro, dummy);
      work(2 + 2 * T, 0, epi, dummy);
    }
    acc[11] += pro;
    acc[12] += epi;
  }
  out[0] = T;
  for (int i = 1; i < 13; ++i) out[i] = nx ? acc[i] / nx : 0.0;
  for (int i = 2; i <= 10; ++i) out[i] /= T > 0 ? T : 1;
}

}  // namespace

extern "C" {

wm_status wm_profile_phases(int32_t on) {
  std::lock_guard<std::mutex> lk(wm::g_pmu);
  wm::g_phases = on != 0;
  if (on) wm::g_pgroups = 0;  // forget the last stamped launch
  return WM_OK;
}

wm_status wm_profile_phases_read(double* out, int32_t n) {
  if (!out || n < 0) return WM_ERR_INVALID_ARG;
  std::vector<unsigned long long> st;
  int groups, nst, T;
  bool nll;
  {
    std::lock_guard<std::mutex> lk(wm::g_pmu);
    groups = wm::g_pgroups;
    nst = wm::g_pnst;
    T = wm::g_pT;
    nll = wm::g_pnll;
    if (groups <= 0 || T <= 0) {
      for (int i = 0; i < n; ++i) out[i] = 0.0;
      return WM_OK;  // no stamped launch
    }
    if (hipDeviceSynchronize() != hipSuccess) return WM_ERR_HIP;
    st.resize((size_t)groups * nst);
    if (hipMemcpy(st.data(), wm::g_pbuf, st.size() * 8, hipMemcpyDeviceToHost) != hipSuccess) return WM_ERR_HIP;
  }
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || khz <= 0)
    return WM_ERR_HIP;
  double res[13];
  phase_summary(st, groups, nst, T, nll, 1e3 / khz, res);
  for (int i = 0; i < n; ++i) out[i] = i < 13 ? res[i] : 0.0;
  return WM_OK;
}

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
