// Return scan over dreamed trajectories: discounted returns, or GAE(lambda)
// with a value baseline (the objective of section 2.2, for the PPO updates
// of sections 2.3 and 4.1).  Both are affine recurrences run backwards in
// time,
//     x_t = a_t + b_t x_{t+1},  x_T = 0,
// with (a_t, b_t) = (r_t, gamma (1 - d_t)) for returns, and
// (r_t + gamma (1 - d_t) V_{t+1} - V_t, gamma lambda (1 - d_t)) for the
// advantages (then returns = advantages + V).
//
// Work split: a thread owns one segment of SEG steps of one trajectory; the
// TPT segments of a trajectory cover a window of TPT * SEG steps, windows are
// taken from the end of the rollout backwards with the value entering each
// window carried over.  In a window a thread
//   1. loads its steps (all loads in flight together),
//   2. folds them into one affine map x_{t0} = S + P x_{t0 + SEG},
//   3. composes the maps of the later segments of its trajectory (a suffix
//      scan over TPT lanes with shuffles) to get the value entering it,
//   4. runs its steps backwards from that value and stores the outputs.
// Lanes are ordered trajectory-fastest (lane = segment * TB + trajectory), so
// that each load touches TB consecutive trajectories of one step.
// Memory-bound: every input is read once and every output written once.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wm_kernels.h"
#include "wm_profile.h"

namespace wm {
namespace {

// steps per thread and window (measured at T = 64, B = 16384: 8 steps 6.7 us,
// 16 steps 7.5 us, 4 steps 8.4 us; shorter segments put more waves in flight)
constexpr int SEG = 8;
constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads) k_returns(const ReturnsBufs R, int tpt) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tb = 64 / tpt;                 // trajectories per wave
  const int seg = lane / tb, bl = lane % tb;
  const int b = (blockIdx.x * (kThreads / 64) + wave) * tb + bl;
  const bool bok = b < R.B;
  const int B = R.B, T = R.T;
  const bool gae = R.values != nullptr;
  const int L = tpt * SEG;                 // steps per window
  float carry = 0.f;                       // x at the step after the window
  for (int end = T; end > 0; end -= L) {   // window [end - L, end)
    const int t0 = end - L + seg * SEG;
    float a[SEG], c[SEG], v[SEG + 1];
    if (gae) {  // V at steps t0 .. t0 + SEG (V has T + 1 rows)
#pragma unroll
      for (int i = 0; i <= SEG; ++i) {
        const int t = t0 + i;
        v[i] = bok && t >= 0 && t <= end ? R.values[(long)t * B + b] : 0.f;
      }
    }
#pragma unroll
    for (int i = 0; i < SEG; ++i) {
      const int t = t0 + i;
      const bool ok = bok && t >= 0 && t < end;
      const float r = ok ? R.rewards[(long)t * B + b] : 0.f;
      const float cont = ok && R.dones[(long)t * B + b] == 0 ? 1.f : 0.f;
      // steps outside the window are the identity map (a = 0, b = 1)
      if (gae) {
        a[i] = ok ? r + R.gamma * cont * v[i + 1] - v[i] : 0.f;
        c[i] = ok ? R.gamma * R.lambda * cont : 1.f;
      } else {
        a[i] = r;
        c[i] = ok ? R.gamma * cont : 1.f;
      }
    }
    // this segment's map x_{t0} = S + P x_{t0+SEG}
    float S = 0.f, P = 1.f;
#pragma unroll
    for (int i = SEG - 1; i >= 0; --i) {
      S = a[i] + c[i] * S;
      P = c[i] * P;
    }
    // suffix scan: F_seg = M_seg o M_seg+1 o ... o M_tpt-1
    float FS = S, FP = P;
    for (int k = 1; k < tpt; k <<= 1) {
      const bool has = seg + k < tpt;
      const int src = has ? lane + k * tb : lane;
      const float oS = __shfl(FS, src), oP = __shfl(FP, src);
      if (has) {
        FS = FS + FP * oS;
        FP = FP * oP;
      }
    }
    // value entering this segment: F_seg+1 applied to the carry
    const bool last = seg + 1 >= tpt;
    const int nsrc = last ? lane : lane + tb;
    const float nS = __shfl(FS, nsrc), nP = __shfl(FP, nsrc);
    float x = last ? carry : nS + nP * carry;
    // the window's value at its first step, for the next window (segment 0)
    const float head = __shfl(FS + FP * carry, bl);
#pragma unroll
    for (int i = SEG - 1; i >= 0; --i) {
      const int t = t0 + i;
      x = a[i] + c[i] * x;
      if (bok && t >= 0 && t < end) {
        const long o = (long)t * B + b;
        if (gae) {
          R.advantages[o] = x;
          R.returns[o] = x + v[i];
        } else {
          R.returns[o] = x;
        }
      }
    }
    carry = head;
  }
}

}  // namespace

hipError_t launch_returns(const ReturnsBufs& R, hipStream_t s) {
  if (R.B <= 0 || R.T <= 0) return hipSuccess;
  const int nseg = (R.T + SEG - 1) / SEG;
  int tpt = 1;
  while (tpt < nseg && tpt < 16) tpt <<= 1;
  const int per_block = (kThreads / 64) * (64 / tpt);
  const unsigned grid = (unsigned)((R.B + per_block - 1) / per_block);
  return launch("returns", k_returns, dim3(grid), dim3(kThreads), 0, s, R, tpt);
}

}  // namespace wm
