// C ABI of libwm: argument checks, workspace carving and dispatch to the HIP
// launchers.  The semantics of each entry point are documented in
// include/wm.h.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <cstdarg>
#include <cstdio>
#include <string>

#include "../../include/wm.h"
#include "wm_kernels.h"

namespace {

thread_local std::string g_err;

wm_status fail(wm_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

wm_status ok() {
  g_err.clear();
  return WM_OK;
}

wm_status hip_fail(hipError_t e, const char* where) {
  return fail(WM_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// Checks the model dims; returns WM_OK and fills the layout.
wm_status check_dims(const wm_dims* d, wm::Layout* L) {
  if (!d) return fail(WM_ERR_INVALID_ARG, "dims is NULL");
  if (d->Z <= 0 || d->H <= 0 || d->A <= 0 || d->K <= 0)
    return fail(WM_ERR_INVALID_ARG, "dims must be positive (Z=%d H=%d A=%d K=%d)", d->Z, d->H,
                d->A, d->K);
  if (d->dtype != WM_FP32 && d->dtype != WM_BF16)
    return fail(WM_ERR_INVALID_ARG, "unknown dtype %d", d->dtype);
  if (d->Z % 8 != 0 || d->Z > 1024)
    return fail(WM_ERR_UNSUPPORTED, "Z=%d: kernels need Z a multiple of 8, at most 1024", d->Z);
  if (d->H % 16 != 0 || d->H > 8192)
    return fail(WM_ERR_UNSUPPORTED, "H=%d: kernels need H a multiple of 16, at most 8192", d->H);
  if (d->K > 8) return fail(WM_ERR_UNSUPPORTED, "K=%d: at most 8 components", d->K);
  if (d->N < 0 || d->L < 0 || (d->N == 0) != (d->L == 0))
    return fail(WM_ERR_INVALID_ARG, "N=%d and L=%d must both be 0 or both positive", d->N, d->L);
  if (d->N == 0 && d->A > 2048)
    return fail(WM_ERR_UNSUPPORTED, "A=%d: at most 2048 actions for a one-level controller", d->A);
  if (d->N > 0 && (int64_t)d->N * d->L != d->A)
    return fail(WM_ERR_INVALID_ARG, "two-level controller: A=%d must equal N*L=%d*%d", d->A, d->N, d->L);
  if (d->N > 0 && (d->N + 1 > 1024 || d->L > 1024))
    return fail(WM_ERR_UNSUPPORTED, "two-level controller: N+1=%d and L=%d must be at most 1024", d->N + 1,
                d->L);
  // the one-hot block (A rows of 4H) is addressed with 32-bit byte offsets
  if ((int64_t)d->A * 4 * d->H * (d->dtype == WM_FP32 ? 4 : 2) >= ((int64_t)1 << 31))
    return fail(WM_ERR_UNSUPPORTED, "A=%d, H=%d: the one-hot block exceeds 2 GiB", d->A, d->H);
  *L = wm::make_layout(d->Z, d->H, d->A, d->K, d->dtype, d->N, d->L);
  return WM_OK;
}

wm_status check_packed(const wm::Layout& L, const void* packed) {
  if (!packed) return fail(WM_ERR_INVALID_ARG, "packed weights pointer is NULL");
  if (reinterpret_cast<uintptr_t>(packed) & 255u)
    return fail(WM_ERR_INVALID_ARG, "packed weights must be 256-byte aligned");
  (void)L;
  return WM_OK;
}

// Reads the status words at the start of a rollout / NLL workspace after the
// stream's work has finished.
wm_status read_status(const void* workspace, hipStream_t s) {
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "waiting for the stream");
  unsigned w[2] = {0u, 0u};
  e = hipMemcpy(w, reinterpret_cast<const unsigned*>(workspace) + wm::kSyncErr, sizeof w,
                hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "reading the workspace status");
  if (w[0]) return fail(WM_ERR_HIP, "a barrier wait of the persistent kernel timed out: the outputs are incomplete");
  if (w[1]) return fail(WM_ERR_INVALID_ARG, "WM_FLAG_CHECK: %u precondition violations in the device data", w[1]);
  return WM_OK;
}

// WM_FLAG_CHECK: zero the status words, run the checks `run` enqueues, wait, read.
template <typename F>
wm_status run_checks(void* workspace, hipStream_t s, F run) {
  unsigned* sync = reinterpret_cast<unsigned*>(workspace);
  hipError_t e = wm::launch_check_zero(sync, s);
  if (e == hipSuccess) e = run(sync);
  if (e != hipSuccess) return hip_fail(e, "WM_FLAG_CHECK");
  return read_status(workspace, s);
}

uint32_t key_lo(uint64_t s) { return (uint32_t)(s & 0xffffffffu); }
uint32_t key_hi(uint64_t s) { return (uint32_t)(s >> 32); }

wm_status rollout_call(const wm_dims* dims, const void* packed, int32_t B, int32_t T,
                     uint32_t traj0, uint32_t step0, const float* z0, const float* h0,
                     const float* c0, uint8_t* done_io, const int32_t* lengths, const uint8_t* valid_mask, uint64_t seed,
                     float tau, uint32_t flags, float* z_out, int32_t* actions, float* rewards,
                     uint8_t* dones, float* h_T, float* c_T, float* h_trace, float* c_trace,
                     void* workspace, size_t workspace_bytes, wm_stream_t stream, bool noalloc) {
  wm::Layout L;
  wm_status st = check_dims(dims, &L);
  if (st != WM_OK) return st;
  if ((st = check_packed(L, packed)) != WM_OK) return st;
  if (B <= 0) return fail(WM_ERR_INVALID_ARG, "B=%d must be positive", B);
  if (T < 0) return fail(WM_ERR_INVALID_ARG, "T=%d must not be negative", T);
  if (!(tau > 0.0f) || !isfinite(tau)) return fail(WM_ERR_INVALID_ARG, "tau must be finite and > 0");
  if (flags & ~(uint32_t)(WM_FLAG_DONE | WM_FLAG_TRACE | WM_FLAG_CHECK | WM_FLAG_SIGMA_TAU |
                          WM_FLAG_STEP_MASK | WM_FLAG_TEST_ABORT))
    return fail(WM_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
  if (!z0 || !valid_mask || !z_out || !actions || !rewards || !dones)
    return fail(WM_ERR_INVALID_ARG, "z0, valid_mask, z_out, actions, rewards, dones are required");
  if (L.N > 0 && (flags & WM_FLAG_STEP_MASK))
    return fail(WM_ERR_UNSUPPORTED, "per-step masks with the two-level controller");
  if ((flags & WM_FLAG_TRACE) && (!h_trace || !c_trace))
    return fail(WM_ERR_INVALID_ARG, "WM_FLAG_TRACE needs h_trace and c_trace");
  if (!aligned16(z0) || !aligned16(z_out))
    return fail(WM_ERR_INVALID_ARG, "z0 and z_out must be 16-byte aligned");
  if ((int64_t)B * (T + 1) > (int64_t)1 << 30)
    return fail(WM_ERR_UNSUPPORTED, "B*(T+1) too large");
  if (T == 0) return ok();
  const size_t need = wm::rollout_workspace(L, B, nullptr, nullptr);
  if (noalloc) {
    if (need > wm::kStaticScratchBytes)
      return fail(WM_ERR_UNSUPPORTED, "wm_rollout_noalloc: B=%d needs %zu bytes of workspace, above the "
                  "%zu-byte static scratch", B, need, wm::kStaticScratchBytes);
    const hipError_t e = wm::static_scratch(&workspace);
    if (e != hipSuccess) return hip_fail(e, "wm_rollout_noalloc: the static scratch");
    workspace_bytes = wm::kStaticScratchBytes;
  }
  if (!workspace || workspace_bytes < need)
    return fail(WM_ERR_WORKSPACE, "rollout workspace needs %zu bytes, got %zu", need, workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(WM_ERR_INVALID_ARG, "workspace must be 256-byte aligned");

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (flags & WM_FLAG_CHECK) {
    // mask bytes: [B, A], [T, B, A] per step, or the two-level xfer and
    // location masks [B, N+1] + [B, N, L]
    const long nmask = L.N > 0 ? (long)B * (L.N + 1) + (long)B * L.N * L.Lc
                               : (long)B * L.A * ((flags & WM_FLAG_STEP_MASK) ? T : 1);
    if ((st = run_checks(workspace, s, [&](unsigned* sync) {
           return wm::launch_check_bytes01(valid_mask, nmask, sync, s);
         })) != WM_OK)
      return st;
  }
  char* ws = reinterpret_cast<char*>(workspace);
  wm::RolloutBufs R{};
  R.B = B; R.T = T; R.traj0 = traj0; R.step0 = step0;
  R.k0 = key_lo(seed); R.k1 = key_hi(seed);
  R.tau = tau; R.flags = flags;
  R.z0 = z0; R.h0 = h0; R.c0 = c0; R.done_io = done_io; R.lengths = lengths; R.mask = valid_mask;
  R.z_out = z_out; R.actions = actions; R.rewards = rewards; R.dones = dones;
  R.h_T = h_T; R.c_T = c_T; R.h_trace = h_trace; R.c_trace = c_trace;
  wm::rollout_workspace(L, B, ws, &R);
  R.preset_err = (flags & WM_FLAG_TEST_ABORT) ? 1u : 0u;
  wm::Packed P{L, packed};
  hipError_t e = wm::launch_rollout(P, R, s);
  if (e != hipSuccess) return hip_fail(e, "wm_rollout");
  if (flags & WM_FLAG_CHECK) return (st = read_status(workspace, s)) == WM_OK ? ok() : st;
  return ok();
}

}  // namespace

extern "C" {

size_t wm_packed_weights_bytes(const wm_dims* dims) {
  wm::Layout L;
  if (check_dims(dims, &L) != WM_OK) return 0;
  return L.total;
}

size_t wm_workspace_bytes(const wm_dims* dims, int32_t B, int32_t T, int32_t which) {
  wm::Layout L;
  if (check_dims(dims, &L) != WM_OK || B <= 0 || T < 0) return 0;
  // sizes the calls refuse need no workspace (and would overflow the sums)
  if ((int64_t)B * (T + 1) > (int64_t)1 << 30) return 0;
  if (which == 3 && (int64_t)B * T > (int64_t)1 << 22) return 0;
  if (which == 0) return wm::rollout_workspace(L, B, nullptr, nullptr);
  if (which == 1) return wm::nll_workspace(L, B, T, nullptr, nullptr);
  if (which == 2) return 0;  // wm_controller_step takes no workspace
  if (which == 3)
    return wm::wm_align256(wm::nll_workspace(L, B, T, nullptr, nullptr)) +
           wm::grad_workspace(L, B, T, nullptr, nullptr);
  return 0;
}

wm_status wm_pack_weights(const wm_dims* dims, const wm_weights* c, void* packed,
                          size_t packed_bytes, wm_stream_t stream) {
  wm::Layout L;
  wm_status st = check_dims(dims, &L);
  if (st != WM_OK) return st;
  if ((st = check_packed(L, packed)) != WM_OK) return st;
  if (!c) return fail(WM_ERR_INVALID_ARG, "weights is NULL");
  if (!c->W_g || !c->b_g || !c->W_m || !c->b_m || !c->w_r || !c->b_r || !c->w_d || !c->b_d ||
      !c->W_c || !c->b_c)
    return fail(WM_ERR_INVALID_ARG, "a canonical weight pointer is NULL");
  if (packed_bytes < L.total)
    return fail(WM_ERR_INVALID_ARG, "packed buffer has %zu bytes, needs %zu", packed_bytes, L.total);
  wm::Packed P{L, packed};
  hipError_t e = wm::launch_pack(P, packed, c->W_g, c->b_g, c->W_m, c->b_m, c->w_r, c->b_r, c->w_d,
                                 c->b_d, c->W_c, c->b_c, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "wm_pack_weights");
  return ok();
}

wm_status wm_controller_step(const wm_dims* dims, const void* packed, int32_t B, uint32_t traj0,
                             const float* z, const float* h, const uint8_t* valid_mask,
                             uint64_t seed, uint32_t step, float* probs, int32_t* action,
                             wm_stream_t stream) {
  wm::Layout L;
  wm_status st = check_dims(dims, &L);
  if (st != WM_OK) return st;
  if ((st = check_packed(L, packed)) != WM_OK) return st;
  if (B <= 0) return fail(WM_ERR_INVALID_ARG, "B=%d must be positive", B);
  if (L.N > 0 && !probs)
    return fail(WM_ERR_INVALID_ARG, "the two-level controller step needs probs [B, N+1+L] (it holds the logits)");
  if (!z || !h || !valid_mask || !action)
    return fail(WM_ERR_INVALID_ARG, "z, h, valid_mask and action are required");
  if (!aligned16(z) || !aligned16(h)) return fail(WM_ERR_INVALID_ARG, "z and h must be 16-byte aligned");
  wm::Packed P{L, packed};
  hipError_t e = wm::launch_controller_step(P, B, traj0, z, h, valid_mask, key_lo(seed),
                                            key_hi(seed), step, probs, action,
                                            reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "wm_controller_step");
  return ok();
}

wm_status wm_rollout(const wm_dims* dims, const void* packed, int32_t B, int32_t T,
                     uint32_t traj0, uint32_t step0, const float* z0, const float* h0,
                     const float* c0, uint8_t* done_io, const int32_t* lengths, const uint8_t* valid_mask, uint64_t seed,
                     float tau, uint32_t flags, float* z_out, int32_t* actions, float* rewards,
                     uint8_t* dones, float* h_T, float* c_T, float* h_trace, float* c_trace,
                     void* workspace, size_t workspace_bytes, wm_stream_t stream) {
  return rollout_call(dims, packed, B, T, traj0, step0, z0, h0, c0, done_io, lengths, valid_mask, seed, tau,
                      flags, z_out, actions, rewards, dones, h_T, c_T, h_trace, c_trace, workspace,
                      workspace_bytes, stream, false);
}

wm_status wm_rollout_noalloc(const wm_dims* dims, const void* packed, int32_t B, int32_t T,
                             uint32_t traj0, uint32_t step0, const float* z0, const float* h0,
                             const float* c0, uint8_t* done_io, const int32_t* lengths, const uint8_t* valid_mask,
                             uint64_t seed, float tau, uint32_t flags, float* z_out,
                             int32_t* actions, float* rewards, uint8_t* dones, float* h_T,
                             float* c_T, float* h_trace, float* c_trace, wm_stream_t stream) {
  return rollout_call(dims, packed, B, T, traj0, step0, z0, h0, c0, done_io, lengths, valid_mask, seed, tau,
                      flags, z_out, actions, rewards, dones, h_T, c_T, h_trace, c_trace, nullptr, 0,
                      stream, true);
}

wm_status wm_nll(const wm_dims* dims, const void* packed, int32_t B, int32_t T, const float* z,
                 const int32_t* actions, const float* rewards, const uint8_t* dones,
                 const int32_t* lengths, uint32_t flags, float* loglik, float* reward_se,
                 float* done_bce, float* means, void* workspace, size_t workspace_bytes,
                 wm_stream_t stream) {
  wm::Layout L;
  wm_status st = check_dims(dims, &L);
  if (st != WM_OK) return st;
  if ((st = check_packed(L, packed)) != WM_OK) return st;
  if (B <= 0) return fail(WM_ERR_INVALID_ARG, "B=%d must be positive", B);
  if (T < 0) return fail(WM_ERR_INVALID_ARG, "T=%d must not be negative", T);
  if (flags & ~(uint32_t)(WM_FLAG_CHECK | WM_FLAG_TEST_ABORT))
    return fail(WM_ERR_INVALID_ARG, "wm_nll: flags 0x%x (only WM_FLAG_CHECK, WM_FLAG_TEST_ABORT)", flags);
  if (!z || !actions || !rewards || !dones || !loglik || !reward_se || !done_bce)
    return fail(WM_ERR_INVALID_ARG, "z, actions, rewards, dones and the three outputs are required");
  if (!aligned16(z)) return fail(WM_ERR_INVALID_ARG, "z must be 16-byte aligned");
  if ((int64_t)B * (T + 1) > (int64_t)1 << 30)
    return fail(WM_ERR_UNSUPPORTED, "B*(T+1) too large");
  if (T == 0) return ok();
  const size_t need = wm::nll_workspace(L, B, T, nullptr, nullptr);
  if (!workspace || workspace_bytes < need)
    return fail(WM_ERR_WORKSPACE, "nll workspace needs %zu bytes, got %zu", need, workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(WM_ERR_INVALID_ARG, "workspace must be 256-byte aligned");

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if ((flags & WM_FLAG_CHECK) && (st = run_checks(workspace, s, [&](unsigned* sync) {
                                    return wm::launch_check_nll(T, B, L.A, actions, dones, lengths, sync, s);
                                  })) != WM_OK)
    return st;
  char* ws = reinterpret_cast<char*>(workspace);
  wm::NllBufs N{};
  N.B = B; N.T = T; N.z = z; N.actions = actions; N.rewards = rewards; N.dones = dones;
  N.lengths = lengths; N.loglik = loglik; N.reward_se = reward_se; N.done_bce = done_bce;
  N.means = means;
  wm::nll_workspace(L, B, T, ws, &N);
  N.preset_err = (flags & WM_FLAG_TEST_ABORT) ? 1u : 0u;
  wm::Packed P{L, packed};
  hipError_t e = wm::launch_nll(P, N, s);
  if (e != hipSuccess) return hip_fail(e, "wm_nll");
  if (flags & WM_FLAG_CHECK) return (st = read_status(workspace, s)) == WM_OK ? ok() : st;
  return ok();
}

wm_status wm_nll_grad(const wm_dims* dims, const void* packed, int32_t B, int32_t T, const float* z,
                      const int32_t* actions, const float* rewards, const uint8_t* dones,
                      const int32_t* lengths, uint32_t flags, float* loss, float* grad_W_g, float* grad_b_g,
                      float* grad_W_m, float* grad_b_m, float* grad_w_r, float* grad_b_r,
                      float* grad_w_d, float* grad_b_d, void* workspace, size_t workspace_bytes,
                      wm_stream_t stream) {
  wm::Layout L;
  wm_status st = check_dims(dims, &L);
  if (st != WM_OK) return st;
  if ((st = check_packed(L, packed)) != WM_OK) return st;
  if (L.dt != 0) return fail(WM_ERR_UNSUPPORTED, "wm_nll_grad serves fp32 weights only");
  if (B <= 0) return fail(WM_ERR_INVALID_ARG, "B=%d must be positive", B);
  if (T < 0) return fail(WM_ERR_INVALID_ARG, "T=%d must not be negative", T);
  if (flags & ~(uint32_t)(WM_FLAG_CHECK | WM_FLAG_TEST_ABORT))
    return fail(WM_ERR_INVALID_ARG, "wm_nll_grad: flags 0x%x (only WM_FLAG_CHECK, WM_FLAG_TEST_ABORT)", flags);
  if (!z || !actions || !rewards || !dones)
    return fail(WM_ERR_INVALID_ARG, "z, actions, rewards and dones are required");
  if (!grad_W_g || !grad_b_g || !grad_W_m || !grad_b_m || !grad_w_r || !grad_b_r || !grad_w_d || !grad_b_d)
    return fail(WM_ERR_INVALID_ARG, "every gradient output is required");
  if (!aligned16(z)) return fail(WM_ERR_INVALID_ARG, "z must be 16-byte aligned");
  if ((int64_t)B * T > (int64_t)1 << 22) return fail(WM_ERR_UNSUPPORTED, "T*B above 2^22");
  if (T == 0) return ok();
  const size_t nb = wm::wm_align256(wm::nll_workspace(L, B, T, nullptr, nullptr));
  const size_t need = nb + wm::grad_workspace(L, B, T, nullptr, nullptr);
  if (!workspace || workspace_bytes < need)
    return fail(WM_ERR_WORKSPACE, "nll_grad workspace needs %zu bytes, got %zu", need, workspace_bytes);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(WM_ERR_INVALID_ARG, "workspace must be 256-byte aligned");

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if ((flags & WM_FLAG_CHECK) && (st = run_checks(workspace, s, [&](unsigned* sync) {
                                    return wm::launch_check_nll(T, B, L.A, actions, dones, lengths, sync, s);
                                  })) != WM_OK)
    return st;
  char* ws = reinterpret_cast<char*>(workspace);
  wm::NllBufs N{};
  N.B = B; N.T = T; N.z = z; N.actions = actions; N.rewards = rewards; N.dones = dones;
  N.lengths = lengths;
  wm::nll_workspace(L, B, T, ws, &N);
  N.preset_err = (flags & WM_FLAG_TEST_ABORT) ? 1u : 0u;
  wm::GradWs G{};
  wm::grad_workspace(L, B, T, ws + nb, &G);
  const wm::GradOut out{loss, grad_W_g, grad_b_g, grad_W_m, grad_b_m, grad_w_r, grad_b_r, grad_w_d, grad_b_d};
  wm::Packed P{L, packed};
  hipError_t e = wm::launch_nll_grad(P, N, G, out, s);
  if (e != hipSuccess) return hip_fail(e, "wm_nll_grad");
  if (flags & WM_FLAG_CHECK) return (st = read_status(workspace, s)) == WM_OK ? ok() : st;
  return ok();
}

wm_status wm_returns(int32_t B, int32_t T, const float* rewards, const uint8_t* dones,
                     const float* values, float gamma, float lambda, float* returns,
                     float* advantages, wm_stream_t stream) {
  if (B < 0 || T < 0) return fail(WM_ERR_INVALID_ARG, "B=%d and T=%d must not be negative", B, T);
  if (!(gamma >= 0.0f && gamma <= 1.0f)) return fail(WM_ERR_INVALID_ARG, "gamma must lie in [0, 1]");
  if (!(lambda >= 0.0f && lambda <= 1.0f)) return fail(WM_ERR_INVALID_ARG, "lambda must lie in [0, 1]");
  if (advantages && !values) return fail(WM_ERR_INVALID_ARG, "advantages need values");
  if ((int64_t)B * (T + 1) > (int64_t)1 << 31)
    return fail(WM_ERR_UNSUPPORTED, "B*(T+1) too large");
  if (B == 0 || T == 0) return ok();
  if (!rewards || !dones || !returns)
    return fail(WM_ERR_INVALID_ARG, "rewards, dones and returns are required");
  if (!aligned4(rewards) || !aligned4(returns) || !aligned4(values) || !aligned4(advantages))
    return fail(WM_ERR_INVALID_ARG, "float arrays must be 4-byte aligned");
  wm::ReturnsBufs R{};
  R.B = B; R.T = T; R.gamma = gamma; R.lambda = lambda;
  R.rewards = rewards; R.dones = dones; R.values = values;
  R.returns = returns; R.advantages = advantages;
  hipError_t e = wm::launch_returns(R, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "wm_returns");
  return ok();
}

wm_status wm_adam_step(int64_t n, float* params, const float* grads, float* m, float* v,
                       int32_t step, float lr, float beta1, float beta2, float eps,
                       wm_stream_t stream) {
  if (n < 0) return fail(WM_ERR_INVALID_ARG, "n=%lld must not be negative", (long long)n);
  if (step < 1) return fail(WM_ERR_INVALID_ARG, "step=%d: Adam steps count from 1", step);
  if (!(lr >= 0.0f) || !isfinite(lr)) return fail(WM_ERR_INVALID_ARG, "lr must be finite and >= 0");
  if (!(beta1 >= 0.0f && beta1 < 1.0f) || !(beta2 >= 0.0f && beta2 < 1.0f))
    return fail(WM_ERR_INVALID_ARG, "beta1 and beta2 must lie in [0, 1)");
  if (!(eps > 0.0f)) return fail(WM_ERR_INVALID_ARG, "eps must be > 0");
  if (n == 0) return ok();
  if (!params || !grads || !m || !v) return fail(WM_ERR_INVALID_ARG, "params, grads, m and v are required");
  if (!aligned16(params) || !aligned16(grads) || !aligned16(m) || !aligned16(v))
    return fail(WM_ERR_INVALID_ARG, "params, grads, m and v must be 16-byte aligned");
  hipError_t e = wm::launch_adam((long)n, params, grads, m, v, step, lr, beta1, beta2, eps,
                                 reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "wm_adam_step");
  return ok();
}

float wm_poly_lr(int32_t epoch, float lr0, float lr_end, int32_t epochs) {
  if (epochs <= 0) return lr_end;
  const double e = epoch < 0 ? 0.0 : (epoch > epochs ? (double)epochs : (double)epoch);
  const double f = 1.0 - e / epochs;
  return (float)(((double)lr0 - lr_end) * f * f + lr_end);
}

wm_status wm_workspace_status(const void* workspace, wm_stream_t stream) {
  if (!workspace) return fail(WM_ERR_INVALID_ARG, "workspace is NULL");
  const wm_status st = read_status(workspace, reinterpret_cast<hipStream_t>(stream));
  return st == WM_OK ? ok() : st;
}

const char* wm_last_error(void) { return g_err.c_str(); }

const char* wm_version(void) { return "libwm 0.1.0 (gfx950)"; }

}  // extern "C"
