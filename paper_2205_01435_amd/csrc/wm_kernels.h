// Launch interface between the C ABI (wm_api.cpp) and the HIP kernels
// (wm_kernels.hip).  Internal to libwm.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/wm.h"
#include "wm_layout.h"

namespace wm {

// Arguments shared by every kernel: the packed weights and their layout.
struct Packed {
  Layout L;
  const void* base;  // device pointer to the packed buffer
};

struct RolloutBufs {
  int B, T;
  uint32_t traj0, step0, k0, k1;  // k0, k1: Philox key words
  float tau;
  uint32_t flags;
  const float *z0, *h0, *c0;
  uint8_t* done_io;
  const int32_t* lengths;  // [B] per-trajectory horizons, or null (T for all)
  const uint8_t* mask;
  float* z_out;
  int32_t* actions;
  float* rewards;
  uint8_t* dones;
  float *h_T, *c_T, *h_trace, *c_trace;
  // workspace
  void* x;             // [2, B, ldx] dtype: activation matrices X_t, X_t+1
  float* c;            // [B, H]
  int32_t* done_state; // [B]
  float* P;            // [32, B, Nc] controller partial logits (persistent kernel) or null
  float* lg;           // [B, Nc] logits of a wide two-level controller, or null
  unsigned* sync;      // kSyncWords barrier and status words, at workspace offset 0
  unsigned preset_err; // initial value of the error word (WM_FLAG_TEST_ABORT)
};

struct NllBufs {
  int B, T;
  const float* z;
  const int32_t* actions;
  const float* rewards;
  const uint8_t* dones;
  const int32_t* lengths;
  float *loglik, *reward_se, *done_bce, *means;
  // workspace
  void* x;       // [T+1, B, ldx] dtype: activation matrices X_0 .. X_T
  float* c;      // [B, H]
  float* part;   // [T*B, NTd]
  float* head;   // [T*B, 2]
  float* wgsum;  // [nwg, 4]
  unsigned* sync;  // kSyncWords barrier and status words, at workspace offset 0
  unsigned preset_err;  // initial value of the error word (WM_FLAG_TEST_ABORT)
  // optional traces of the persistent recurrence (training gradient): gate
  // activations (i, f, tanh g, o) [T, B, 4H] in the packed gate order, and
  // c_{t+1} at [t+1] of [T+1, B, H]
  float* g_trace;
  float* c_trace;
};

// Barrier and status words (zeroed by the init kernels) at offset 0 of the
// rollout and NLL workspaces: the persistent kernels' group counters at
// 64 x and placement flags at 64 (8 + x); the error word (a barrier wait
// timed out) and the WM_FLAG_CHECK violation count.
constexpr int kSyncWords = 64 * 17;
constexpr int kSyncErr = 64 * 16;
constexpr int kSyncViol = 64 * 16 + 1;

// Workspace sizes; with a non-null `ws` the workspace pointers of the
// buffer struct are also set (ws must be 256-byte aligned).
size_t rollout_workspace(const Layout& L, int B, char* ws, RolloutBufs* R);
size_t nll_workspace(const Layout& L, int B, int T, char* ws, NllBufs* N);

hipError_t launch_pack(const Packed& P, void* packed, const float* W_g, const float* b_g,
                       const float* W_m, const float* b_m, const float* w_r, const float* b_r,
                       const float* w_d, const float* b_d, const float* W_c, const float* b_c,
                       hipStream_t s);

hipError_t launch_controller_step(const Packed& P, int B, uint32_t traj0, const float* z,
                                  const float* h, const uint8_t* mask, uint32_t k0, uint32_t k1,
                                  uint32_t step, float* probs, int32_t* action, hipStream_t s);

hipError_t launch_rollout(const Packed& P, const RolloutBufs& R, hipStream_t s);

// WM_FLAG_CHECK passes: zero the two status words, then count violations
// of the device-data preconditions into sync[kSyncViol].
hipError_t launch_check_zero(unsigned* sync, hipStream_t s);
// bytes of p[0 .. n) other than 0 and 1
hipError_t launch_check_bytes01(const uint8_t* p, long n, unsigned* sync, hipStream_t s);
// actions of steps t < lengths[b] outside [0, A) u {-1, -2}; dones other than 0, 1
hipError_t launch_check_nll(int T, int B, int A, const int32_t* actions, const uint8_t* dones,
                            const int32_t* lengths, unsigned* sync, hipStream_t s);

hipError_t launch_nll(const Packed& P, const NllBufs& N, hipStream_t s);

// Persistent single-launch kernels (wm_persist.hip) for small fp32 batches.
// The launchers return hipErrorNotSupported when the dims, the batch or the
// device are outside what they serve (or WM_PERSISTENT=0 is set).
size_t persist_partial_bytes(const Layout& L, int B);  // 0 if not served
bool persist_usable(const Layout& L, int B, bool nll);
hipError_t launch_rollout_persist(const Packed& P, const RolloutBufs& R, hipStream_t s);
hipError_t launch_nll_persist(const Packed& P, const NllBufs& N, hipStream_t s);

// The static device scratch of wm_rollout_noalloc (wm_noalloc.hip): its
// device address on the current device, looked up once per device.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
hipError_t static_scratch(void** ptr);

// Return scan over B trajectories of T steps (wm_returns.hip).
struct ReturnsBufs {
  int B, T;
  float gamma, lambda;
  const float* rewards;  // [T, B]
  const uint8_t* dones;  // [T, B]
  const float* values;   // [T+1, B] or null
  float* returns;        // [T, B]
  float* advantages;     // [T, B] or null (values given)
};
hipError_t launch_returns(const ReturnsBufs& R, hipStream_t s);

// World-model training step: gradient of the summed NLL means (fp32).
struct GradWs {  // workspace after the NLL pass's own
  float *G, *Cs, *M, *dG, *dhh, *dh, *dc;
  float *dWgT, *dWa, *dWm, *dbg, *dbm, *part, *apart, *split, *nsum, *fwd;
};
struct GradOut {  // canonical gradients; loss (nullable): the summed means
  float *loss, *W_g, *b_g, *W_m, *b_m, *w_r, *b_r, *w_d, *b_d;
};
size_t grad_workspace(const Layout& L, int B, int T, char* ws, GradWs* G);
hipError_t launch_nll_grad(const Packed& P, NllBufs N, const GradWs& G, const GradOut& out, hipStream_t s);

// Adam step on n fp32 parameters, in place (wm_optim.hip).
hipError_t launch_adam(long n, float* p, const float* g, float* m, float* v, int step, float lr,
                       float beta1, float beta2, float eps, hipStream_t s);

}  // namespace wm
