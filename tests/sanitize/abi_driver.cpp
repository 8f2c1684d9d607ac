// Host-side driver of the C ABI for sanitizer builds (AddressSanitizer +
// UndefinedBehaviorSanitizer, or ThreadSanitizer): every call here fails
// validation, takes a documented no-op path, or touches only the host-side
// registries, so no call reaches the GPU and the driver runs on a machine
// without one.  Fake device pointers are never dereferenced: validation
// rejects the call first.  Exit status 0 when every expectation holds.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

#include "wm.h"

static int g_failures = 0;

#define EXPECT(cond)                                                               \
  do {                                                                             \
    if (!(cond)) {                                                                 \
      std::fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
      ++g_failures;                                                                \
    }                                                                              \
  } while (0)

static wm_dims dims(int Z, int H, int A, int K, int dt = WM_FP32, int N = 0, int L = 0) {
  wm_dims d;
  d.Z = Z; d.H = H; d.A = A; d.K = K; d.dtype = dt; d.N = N; d.L = L;
  return d;
}

template <typename T>
static T* fake(uintptr_t a) { return reinterpret_cast<T*>(a); }

static void sizes() {
  EXPECT(std::strstr(wm_version(), "libwm") != nullptr);
  const wm_dims ok = dims(64, 512, 64, 5);
  EXPECT(wm_packed_weights_bytes(&ok) > 0);
  EXPECT(wm_packed_weights_bytes(nullptr) == 0);
  const wm_dims bad[] = {dims(0, 16, 4, 2), dims(8, 16, 4, 0), dims(6, 16, 4, 2), dims(8, 24, 4, 2),
                         dims(8, 16, 4, 9), dims(8, 16, 4096, 2), dims(8, 16, 4, 2, 7),
                         dims(8, 16, 6, 2, WM_FP32, 2, 0), dims(8, 16, 6, 2, WM_FP32, 2, 4),
                         dims(8, 16, 2050 * 3, 2, WM_FP32, 2050, 3), dims(1032, 16, 4, 2),
                         dims(8, 8208, 4, 2), dims(8, 8192, 57600, 2, WM_BF16, 288, 200),
                         dims(-8, -16, -4, -2)};
  for (const wm_dims& d : bad) {
    EXPECT(wm_packed_weights_bytes(&d) == 0);
    EXPECT(wm_workspace_bytes(&d, 16, 4, 0) == 0);
    EXPECT(std::strlen(wm_last_error()) > 0);
  }
  // the paper's largest two-level action space is supported
  const wm_dims two = dims(64, 512, 57600, 5, WM_BF16, 288, 200);
  EXPECT(wm_packed_weights_bytes(&two) > 0);
  for (int which = -2; which <= 5; ++which)
    for (int B : {0, 1, 7, 256, 4096, 1 << 20})
      for (int T : {0, 1, 50, 1000}) {
        const size_t n = wm_workspace_bytes(&ok, B, T, which);
        if (B == 0 || which < 0 || which > 3 || which == 2) EXPECT(n == 0);
        (void)n;
      }
  EXPECT(wm_workspace_bytes(&ok, -1, 4, 0) == 0);
  EXPECT(wm_workspace_bytes(&ok, 4, -1, 0) == 0);
  EXPECT(wm_workspace_bytes(&ok, 1 << 30, 1 << 30, 1) == 0);  // beyond the size checks
  for (int e : {-5, 0, 1, 2500, 4999, 5000, 7000}) EXPECT(std::isfinite(wm_poly_lr(e, 3e-3f, 1e-5f, 5000)));
  EXPECT(std::isfinite(wm_poly_lr(3, 1e-3f, 1e-4f, 0)));
}

static void controller() {
  const wm_dims d = dims(8, 16, 4, 2);
  float* f = fake<float>(4096);
  uint8_t* m = fake<uint8_t>(4096);
  int32_t* a = fake<int32_t>(4096);
  EXPECT(wm_controller_step(nullptr, f, 4, 0, f, f, m, 1, 0, nullptr, a, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_controller_step(&d, nullptr, 4, 0, f, f, m, 1, 0, nullptr, a, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_controller_step(&d, fake<float>(4112), 4, 0, f, f, m, 1, 0, nullptr, a, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_controller_step(&d, f, 0, 0, f, f, m, 1, 0, nullptr, a, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_controller_step(&d, f, 4, 0, nullptr, f, m, 1, 0, nullptr, a, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_controller_step(&d, f, 4, 0, f, f, nullptr, 1, 0, nullptr, a, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_controller_step(&d, f, 4, 0, f, f, m, 1, 0, nullptr, nullptr, nullptr) == WM_ERR_INVALID_ARG);
  // the two-level controller needs its factored probabilities
  const wm_dims t = dims(8, 16, 6, 2, WM_FP32, 2, 3);
  EXPECT(wm_controller_step(&t, f, 4, 0, f, f, m, 1, 0, nullptr, a, nullptr) == WM_ERR_INVALID_ARG);
}

static wm_status rollout(const wm_dims* d, int B, int T, float tau, uint32_t flags, uintptr_t z0 = 4096,
                         uintptr_t packed = 4096, size_t ws_bytes = 0, bool noalloc = false,
                         uintptr_t trace = 0) {
  float* p = fake<float>(4096);
  uint8_t* m = fake<uint8_t>(4096);
  int32_t* a = fake<int32_t>(4096);
  float* tr = trace ? fake<float>(trace) : nullptr;
  if (noalloc)
    return wm_rollout_noalloc(d, fake<void>(packed), B, T, 0, 0, fake<float>(z0), nullptr, nullptr, nullptr,
                              nullptr, m, 1, tau, flags, p, a, p, m, nullptr, nullptr, tr, tr, nullptr);
  return wm_rollout(d, fake<void>(packed), B, T, 0, 0, fake<float>(z0), nullptr, nullptr, nullptr, nullptr, m, 1,
                    tau, flags, p, a, p, m, nullptr, nullptr, tr, tr, fake<void>(4096), ws_bytes, nullptr);
}

static void rollouts() {
  const wm_dims d = dims(8, 16, 4, 2);
  for (bool na : {false, true}) {
    EXPECT(rollout(&d, 4, 3, 1.f, 1, 0, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 4, 3, 0.f, 1, 4096, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 4, 3, NAN, 1, 4096, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 4, 3, INFINITY, 1, 4096, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 0, 3, 1.f, 1, 4096, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 4, -1, 1.f, 1, 4096, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 4, 3, 1.f, 32, 4096, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 4, 3, 1.f, 3, 4096, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 4, 3, 1.f, 1, 4100, 4096, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 4, 3, 1.f, 1, 4096, 4112, 0, na) == WM_ERR_INVALID_ARG);
    EXPECT(rollout(&d, 1 << 20, 2000, 1.f, 1, 4096, 4096, 0, na) == WM_ERR_UNSUPPORTED);
    // T = 0 is a no-op that touches nothing
    EXPECT(rollout(&d, 4, 0, 1.f, 1 | WM_FLAG_TRACE, 4096, 4096, 0, na, 4096) == WM_OK);
    EXPECT(std::strlen(wm_last_error()) == 0);
  }
  for (uint32_t f : {WM_FLAG_CHECK, WM_FLAG_STEP_MASK, WM_FLAG_SIGMA_TAU, WM_FLAG_TEST_ABORT})
    EXPECT(rollout(&d, 4, 3, 1.f, 1 | f) == WM_ERR_WORKSPACE);
  EXPECT(rollout(&d, 4, 3, 1.f, 1, 4096, 4096, wm_workspace_bytes(&d, 4, 3, 0) - 1) == WM_ERR_WORKSPACE);
  const wm_dims t = dims(8, 16, 6, 2, WM_FP32, 2, 3);
  EXPECT(rollout(&t, 4, 3, 1.f, 1 | WM_FLAG_STEP_MASK) == WM_ERR_UNSUPPORTED);
  // the no-allocation variant refuses workspaces beyond its static scratch
  const wm_dims big = dims(128, 1024, 256, 8, WM_BF16);
  EXPECT(rollout(&big, 1 << 18, 64, 1.f, 1, 4096, 4096, 0, true) == WM_ERR_UNSUPPORTED);
  EXPECT(std::strstr(wm_last_error(), "static scratch") != nullptr);
}

static void nll_and_grad() {
  const wm_dims d = dims(8, 16, 4, 2);
  float* p = fake<float>(4096);
  int32_t* a = fake<int32_t>(4096);
  uint8_t* m = fake<uint8_t>(4096);
  void* w = fake<void>(4096);
  EXPECT(wm_nll(&d, w, 4, 3, nullptr, a, p, m, nullptr, 0, p, p, p, nullptr, w, 0, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_nll(&d, w, 4, 3, p, a, p, m, nullptr, 0, p, p, p, nullptr, w, 0, nullptr) == WM_ERR_WORKSPACE);
  EXPECT(wm_nll(&d, w, 4, 3, p, a, p, m, nullptr, WM_FLAG_DONE, p, p, p, nullptr, w, 0, nullptr) ==
         WM_ERR_INVALID_ARG);
  EXPECT(wm_nll(&d, w, 4, 0, p, a, p, m, nullptr, 0, p, p, p, nullptr, w, 0, nullptr) == WM_OK);
  EXPECT(wm_nll(&d, w, -4, 3, p, a, p, m, nullptr, 0, p, p, p, nullptr, w, 0, nullptr) == WM_ERR_INVALID_ARG);
  auto grad = [&](const wm_dims* dd, int B, int T, float* z, float* out, uint32_t flags) {
    return wm_nll_grad(dd, w, B, T, z, a, p, m, nullptr, flags, nullptr, out, p, p, p, p, p, p, p, w, 0, nullptr);
  };
  EXPECT(grad(&d, 4, 3, nullptr, p, 0) == WM_ERR_INVALID_ARG);
  EXPECT(grad(&d, 4, 3, p, nullptr, 0) == WM_ERR_INVALID_ARG);
  EXPECT(grad(&d, 4, 3, fake<float>(4100), p, 0) == WM_ERR_INVALID_ARG);
  EXPECT(grad(&d, 0, 3, p, p, 0) == WM_ERR_INVALID_ARG);
  EXPECT(grad(&d, 4, 3, p, p, WM_FLAG_TRACE) == WM_ERR_INVALID_ARG);
  EXPECT(grad(&d, 1 << 12, 1 << 11, p, p, 0) == WM_ERR_UNSUPPORTED);
  const wm_dims b = dims(8, 16, 4, 2, WM_BF16);
  EXPECT(grad(&b, 4, 3, p, p, 0) == WM_ERR_UNSUPPORTED);
  EXPECT(grad(&d, 4, 3, p, p, 0) == WM_ERR_WORKSPACE);
  EXPECT(grad(&d, 4, 0, p, p, 0) == WM_OK);
}

static void others() {
  float* p = fake<float>(4096);
  uint8_t* m = fake<uint8_t>(4096);
  EXPECT(wm_pack_weights(nullptr, nullptr, p, 0, nullptr) == WM_ERR_INVALID_ARG);
  const wm_dims d = dims(8, 16, 4, 2);
  EXPECT(wm_pack_weights(&d, nullptr, p, 1 << 20, nullptr) == WM_ERR_INVALID_ARG);
  wm_weights w;
  std::memset(&w, 0, sizeof w);
  EXPECT(wm_pack_weights(&d, &w, p, 1 << 20, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_returns(-1, 3, p, m, p, 0.99f, 0.95f, p, p, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_returns(4, 3, p, m, p, 1.5f, 0.95f, p, p, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_returns(4, 3, nullptr, m, p, 0.99f, 0.95f, p, p, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_returns(4, 0, p, m, p, 0.99f, 0.95f, p, p, nullptr) == WM_OK);
  EXPECT(wm_adam_step(-1, p, p, p, p, 1, 1e-3f, 0.9f, 0.999f, 1e-8f, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_adam_step(16, nullptr, p, p, p, 1, 1e-3f, 0.9f, 0.999f, 1e-8f, nullptr) == WM_ERR_INVALID_ARG);
  EXPECT(wm_adam_step(0, p, p, p, p, 1, 1e-3f, 0.9f, 0.999f, 1e-8f, nullptr) == WM_OK);
  EXPECT(wm_workspace_status(nullptr, nullptr) == WM_ERR_INVALID_ARG);
  // profile registry: no launch has been recorded, so no event is touched
  EXPECT(wm_profile_read("gates", nullptr, nullptr) == WM_ERR_INVALID_ARG);
  std::string longp(10000, 'g');
  EXPECT(wm_profile_enable(longp.c_str()) == WM_OK);
  EXPECT(wm_profile_enable("") == WM_OK);
  double ms = -1.0;
  int64_t n = -1;
  EXPECT(wm_profile_read(nullptr, &ms, &n) == WM_OK && ms == 0.0 && n == 0);
  EXPECT(wm_profile_read("mdn", &ms, &n) == WM_OK && n == 0);
  EXPECT(wm_profile_reset() == WM_OK);
  EXPECT(wm_profile_enable(nullptr) == WM_OK);
  // phase timing: nothing stamped yet, so the read touches no device
  double ph[16];
  for (double& v : ph) v = -1.0;
  EXPECT(wm_profile_phases(1) == WM_OK);
  EXPECT(wm_profile_phases_read(ph, 16) == WM_OK && ph[0] == 0.0 && ph[15] == 0.0);
  EXPECT(wm_profile_phases_read(nullptr, 4) == WM_ERR_INVALID_ARG);
  EXPECT(wm_profile_phases_read(ph, -1) == WM_ERR_INVALID_ARG);
  EXPECT(wm_profile_phases(0) == WM_OK);
}

// Several threads at once: the last-error string is per thread and the
// profile registry is guarded.
static void threads() {
  std::vector<std::thread> th;
  int fails[8] = {0};
  for (int i = 0; i < 8; ++i)
    th.emplace_back([i, &fails] {
      const wm_dims d = dims(8, 16, 4, 2);
      for (int r = 0; r < 200; ++r) {
        const int B = -(i * 1000 + r) - 1;  // a distinct bad B per thread and round
        float* p = fake<float>(4096);
        uint8_t* m = fake<uint8_t>(4096);
        int32_t* a = fake<int32_t>(4096);
        if (wm_controller_step(&d, p, B, 0, p, p, m, 1, 0, nullptr, a, nullptr) != WM_ERR_INVALID_ARG) ++fails[i];
        char want[64];
        std::snprintf(want, sizeof want, "B=%d", B);
        if (!std::strstr(wm_last_error(), want)) ++fails[i];
        if (r % 16 == 0) {
          (void)wm_profile_enable(i % 2 ? "gates" : nullptr);
          double ms;
          int64_t n;
          if (wm_profile_read(nullptr, &ms, &n) != WM_OK) ++fails[i];
          (void)wm_profile_reset();
        }
      }
    });
  for (auto& t : th) t.join();
  for (int i = 0; i < 8; ++i) EXPECT(fails[i] == 0);
  (void)wm_profile_enable(nullptr);
}

int main(int argc, char** argv) {
  const bool threads_only = argc > 1 && std::strcmp(argv[1], "threads") == 0;
  if (!threads_only) {
    sizes();
    controller();
    rollouts();
    nll_and_grad();
    others();
  }
  threads();
  std::printf("abi driver: %d failures\n", g_failures);
  return g_failures ? 1 : 0;
}
