// Persistent kernels of libwm for small batches (fp32) on gfx950 (MI355X):
// one launch runs every step of a dream rollout, or every step of the NLL
// pass's teacher-forced recurrence.
//
// Rows are split over the eight XCDs: XCD x owns rows [x*Bx, (x+1)*Bx) and
// its 32 work-groups (one per CU; blockIdx % 8 selects the XCD) step those
// trajectories together.  Trajectories of different XCDs never exchange
// data, so every barrier is local to one XCD: a counter in that XCD's L2,
// producers wait for their stores to reach the L2 (vmcnt), and everything a
// work-group reads that another one wrote during the call is read with
// device-coherent loads (sc1: past the CU's L1, served by the shared L2), so
// no cache has to be invalidated and the weights stay in the L2.  That costs
// about 0.9 us per barrier on the MI355X, where a kernel boundary costs
// about 4.5 us and a barrier with agent-scope fences 4-7 us.  Each
// work-group checks its hardware XCD id at the start; if any member of a
// group is not on the group's XCD, the group uses agent-scope fences
// instead, so results never depend on the placement.
//
// Each work-group owns NBC blocks of four hidden units (16 gate rows each).
// The gate weights of those rows stay in registers for the whole call (the
// A operand of the MFMAs), and each lane keeps the cell state of the
// (unit, row) pairs it owns in registers.  Per dream step t, two phases
// separated by XCD barriers:
//   gates(t)  X_t of the XCD's rows staged in LDS (LDS-DMA, four chunks so
//             that the MFMAs start on the first), gate GEMM against the
//             register weights.  Under the staging loads, the owner of each
//             row (work-group m % 32 for row m) makes that row's controller
//             decision: logits = W_c,z z_t (vector FMAs against W_c in the
//             L2) + the h part and the bias (from mdn(t-1)), masked
//             Gumbel-max, the reward and done of transition t-1, freeze
//             logic; it writes the row's outputs, then a per-row flag
//             (t + 1) once they have reached the L2.  Before the LSTM cell
//             every work-group waits (bounded) for the flags of the XCD's
//             rows and reads their actions.  LSTM cell with the chosen
//             action's one-hot column, h_{t+1} into X_{t+1};
//   mdn(t)    (group of four latent dims, 16-row block) tiles, K split over
//             the four waves and summed in LDS, component pick, Box-Muller
//             draw, z_{t+1} to z_out and X_{t+1}; further tiles (or, when
//             the tiles do not fit one round of work-groups, the first
//             tiles themselves) compute the next step's controller h part
//             W_c,h h_{t+1} + b_c into Lh (rows A and A+1 of W_c are the
//             reward and done heads).
// The barriers are split: a work-group arrives, draws the random numbers of
// the next phase (the mixture noise of its mdn tile, the controller's
// Gumbel noise), and then waits, so that the draws fill the barrier's
// latency.
// The NLL recurrence runs gates(t) only, one barrier per step; the mixture
// head then runs once over all T*B rows (wm_kernels.hip).
// Every wait is bounded: a wait that times out raises an error word that
// every other wait polls, and all work-groups leave.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdlib>
#include <cstring>

#include "wm_device.h"
#include "wm_kernels.h"
#include "wm_layout.h"
#include "wm_profile.h"

namespace wm {
namespace {

constexpr int kGroups = 8;     // XCDs
constexpr int kMembers = 32;   // work-groups (CUs) per XCD
constexpr int kGrid = kGroups * kMembers;
constexpr int kMaxS = 36;      // register-resident MFMA K slices per wave (4 chunks of 9)
constexpr int kMaxQ = 6;       // mixture output blocks per latent-dim group (K <= 8)
constexpr int kMaxMS = 8;      // mixture-head K slices per wave (H <= 512)
constexpr unsigned kSpinLimit = 1u << 22;

struct PArgs {
  const float *Wg, *WaT, *bg, *Wm, *bm, *Wc, *bc;
  int Z, H, A, K, Q, Nc, ldk, ldh, ldx;
  int B, T, Bx;
  uint32_t k0, k1, traj0, step0;
  float tau;
  float sig;  // scale of the normal deviate (sqrt(tau) with the sigma temperature, else 1)
  int use_done, wat_lds, mres;
  float* X;             // rollout [2, B, ldx]; NLL [T+1, B, ldx]
  float* c;             // [B, H]: initial cell state in, final state out (rollout)
  int32_t* done_state;  // [B]
  const int32_t* lengths;  // [B] per-trajectory horizons, or null
  float* Lh;            // [B, Nc] controller logits' h part + bias (rollout)
  unsigned* flags;      // [B] step t's action of row m is written once flags[m] > t (rollout)
  unsigned* sync;       // kSyncWords words, zero at launch
  const uint8_t* mask;  // [B, A], or [T, B, A] with step_mask
  int step_mask;
  float* z_out;         // [T+1, B, Z]
  int32_t* actions;     // [T, B]: rollout output, NLL input
  float* rewards;
  uint8_t* dones;
  float *h_trace, *c_trace;  // [T+1, B, H] or null (each on its own)
  float* g_trace;            // NLL: gate activations [T, B, 4H] or null
  // LDS carve-up (bytes)
  int off_red, off_rows, off_wat, off_mdn, off_ctl, off_flags, off_mres;
  // controller: Nc / 16 logit blocks; the h-part blocks run as tiles of
  // their own in mdn(t) (1) or inside the first mixture tiles (0)
  int ncb, ctl_sep;
  // phase timing (measurement runs; null otherwise): nst device-clock
  // stamps per work-group, [blockIdx][nst]
  unsigned long long* stamps;
  int nst;
};

// sync words: group counters at 64*x, placement flags at 64*(8+x), error at 64*16
__device__ __forceinline__ unsigned* sync_ctr(const PArgs& p, int x) { return p.sync + 64 * x; }
__device__ __forceinline__ unsigned* sync_flag(const PArgs& p, int x) { return p.sync + 64 * (8 + x); }
__device__ __forceinline__ unsigned* sync_err(const PArgs& p) { return p.sync + 64 * 16; }

__device__ __forceinline__ unsigned xcc_id() { return __builtin_amdgcn_s_getreg((3 << 11) | 20) & 15u; }

struct GroupSync {
  unsigned* ctr;
  unsigned* err;
  unsigned n;  // barriers passed
  bool agent;  // members not all on one XCD: agent-scope fences
  unsigned long long* st;  // this work-group's phase stamps, or null
  int nst;
};

// Phase stamp i of this work-group: the constant-rate device clock, written
// by the calling lane with a vector store.  Slot 0 is the kernel's start,
// 2b-1 and 2b the arrival at and release from barrier b (1, 2, ...), nst-1
// the end.
__device__ __forceinline__ void phase_stamp(unsigned long long* st, int nst, int i) {
  if (!st) return;
  const unsigned long long v = __builtin_amdgcn_s_memrealtime();
  const rsrc_t r = make_rsrc(st, (uint32_t)nst * 8u);
  bstore8(r, (uint32_t)i * 8u, make_uint2((uint32_t)v, (uint32_t)(v >> 32)));
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// Barrier of the 32 work-groups of one XCD, in two halves: group_arrive
// publishes this work-group's stores and counts it in; group_wait waits for
// the other 31.  Work between the two may touch only registers and this
// work-group's own LDS.  group_wait returns false if the group must stop (a
// wait timed out here or elsewhere).
__device__ __forceinline__ void group_arrive(GroupSync& gs) {
  if (gs.agent) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  else asm volatile("s_waitcnt vmcnt(0)" : : : "memory");  // this wave's stores reached L2
  __syncthreads();
  ++gs.n;
  if (threadIdx.x == 0) {
    phase_stamp(gs.st, gs.nst, 2 * (int)gs.n - 1);
    __hip_atomic_fetch_add(gs.ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__device__ __forceinline__ bool group_wait(GroupSync& gs, volatile int* flag) {
  if (threadIdx.x == 0) {
    int ok = 1;
    const unsigned target = gs.n * kMembers;
    unsigned spins = 0;
    while ((int)(__hip_atomic_load(gs.ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - target) < 0) {
      if ((++spins & 63u) == 0) {
        if (__hip_atomic_load(gs.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
          ok = 0;
          break;
        }
        if (spins >= kSpinLimit) {
          __hip_atomic_fetch_or(gs.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          ok = 0;
          break;
        }
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (gs.agent) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    phase_stamp(gs.st, gs.nst, 2 * (int)gs.n);
    *flag = ok;
  }
  __syncthreads();
  return *flag != 0;
}

__device__ __forceinline__ bool group_sync(GroupSync& gs, volatile int* flag) {
  group_arrive(gs);
  return group_wait(gs, flag);
}
#pragma clang diagnostic pop

// Device-coherent (sc1) reads of data other work-groups wrote during the
// call: they bypass this CU's L1, which may still hold an older copy of the
// line, and are served by the XCD's L2.
__device__ __forceinline__ uint32_t cload4(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 16);
}
__device__ __forceinline__ uint4 cload16(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 16));
}
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// dma16 with the device-coherent policy
__device__ __forceinline__ void cdma16(u32x4 rs, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen sc1 lds"
               :
               : "s"(lds), "v"(voff), "s"(rs)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Issue v (0..3) of a 16-wide fp32 K slice (the four issues of Mfma<float>::step).
__device__ __forceinline__ void mfma4(f32x4& acc, const uint4& a, const uint4& b, int v) {
  const uint32_t av = v == 0 ? a.x : v == 1 ? a.y : v == 2 ? a.z : a.w;
  const uint32_t bv = v == 0 ? b.x : v == 1 ? b.y : v == 2 ? b.z : b.w;
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(av), __uint_as_float(bv), acc, 0, 0, 0);
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const char*)p);
}

// ---------------------------------------------------------------------------
// Per-work-group state that lives across steps.
// ---------------------------------------------------------------------------
template <int RB, int NBC>
struct GateState {
  static constexpr int KSPLIT = 4 / NBC;
  uint4 wr[kMaxS];  // gate weights: rows 16 blk + r16, K slices sl0 .. sl0+nper-1
  float4 bias;      // b_g of this lane's unit (owner waves)
  float cst[RB];    // cell state of (unit, row 16 rb + r16) (owner waves)
};

// ---------------------------------------------------------------------------
// Controller decisions (rollout).  Row m of an XCD (m < 64) is owned by
// work-group m % 32 of the XCD, which decides its action at the start of
// gates(t), while its staging loads are in flight: logits = W_c,z q(z_t) (one
// thread per action, W_c's z columns from L2) + Lh (the h part and the bias,
// written by mdn(t-1)), plus the Gumbel noise drawn at the barrier; the best
// valid action, lowest index on ties; then the bookkeeping of transition t-1
// and step t.  The owner writes the action and then the row's flag (t + 1);
// every work-group waits for the flags of the XCD's rows only before its
// cell epilogue, which needs the actions.
// ---------------------------------------------------------------------------
constexpr int kMaxOwn = 2;  // rows per work-group: 64 rows per XCD at most
// Row m's flag after its decision of step t: (t + 1) << kFlagShift |
// (action + 1), so that the action travels in the word that announces it
// and no ordering between two stores is needed (actions are below 1023).
constexpr int kFlagShift = 10;
__device__ __forceinline__ uint32_t row_flag(int t, int act) {
  return ((uint32_t)(t + 1) << kFlagShift) | (uint32_t)(act + 1);
}

// One step of the wave's (score, action) argmax: merge with the pair that
// the DPP pattern CTRL brings in (none: an empty pair).  The merge keeps the
// higher score, the lower action on equal scores, and ignores empty pairs
// (action < 0), so it is idempotent and any covering order gives the same
// result as a butterfly.
template <int CTRL, int ROWM>
__device__ __forceinline__ void argmax_dpp(float& best, int& bi) {
  const float ob = __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(-INFINITY), __float_as_int(best), CTRL, ROWM, 0xf, false));
  const int oi = __builtin_amdgcn_update_dpp(-1, bi, CTRL, ROWM, 0xf, false);
  if (oi >= 0 && (bi < 0 || ob > best || (ob == best && oi < bi))) {
    best = ob;
    bi = oi;
  }
}

// Argmax of (best, bi) over the 64 lanes, lowest action on ties, in every
// lane: row shifts by 1, 2, 4 and 8 leave each row's result in its lane 15,
// the row broadcasts 15 and 31 carry them to lane 63, which is read out.
// (Cross-lane moves on the DPP path instead of 12 dependent LDS-crossbar
// shuffles.)
__device__ __forceinline__ void wave_argmax(float& best, int& bi) {
  argmax_dpp<0x111, 0xf>(best, bi);  // row_shr:1
  argmax_dpp<0x112, 0xf>(best, bi);  // row_shr:2
  argmax_dpp<0x114, 0xf>(best, bi);  // row_shr:4
  argmax_dpp<0x118, 0xf>(best, bi);  // row_shr:8
  argmax_dpp<0x142, 0xa>(best, bi);  // row_bcast:15 into rows 1 and 3
  argmax_dpp<0x143, 0xc>(best, bi);  // row_bcast:31 into rows 2 and 3
  best = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(best), 63));
  bi = __builtin_amdgcn_readlane(bi, 63);
}

struct CtrlLane {
  float gum[kMaxOwn];  // thread a's Gumbel noise for action a of each owned row; -inf: not valid
  float ud[kMaxOwn];   // the stream-3 uniform of transition t-1 of each owned row
};

__device__ __forceinline__ int* row_act(const PArgs& p, char* lds) { return reinterpret_cast<int*>(lds + p.off_rows); }
__device__ __forceinline__ int* row_done(const PArgs& p, char* lds) { return row_act(p, lds) + 64; }
__device__ __forceinline__ int* row_prev(const PArgs& p, char* lds) { return row_act(p, lds) + 128; }
__device__ __forceinline__ int* row_len(const PArgs& p, char* lds) { return row_act(p, lds) + 192; }

// The random numbers of step t for this work-group's rows (drawn while it
// waits at a barrier): thread a takes action a's Gumbel score (-inf where
// the action is not valid), and the done uniforms of transition t-1.
// t == T: the done uniforms only.
__device__ __forceinline__ void ctrl_noise(const PArgs& p, CtrlLane& cl, int t, int r0, int nrows) {
  const int a = threadIdx.x, s = blockIdx.x >> 3;
  const Rng rng{p.k0, p.k1};
  const uint32_t step = p.step0 + (uint32_t)t;
#pragma unroll
  for (int o = 0; o < kMaxOwn; ++o) {
    const int ml = s + kMembers * o;
    cl.gum[o] = -INFINITY;
    cl.ud[o] = 0.f;
    if (ml >= nrows) continue;
    const uint32_t traj = p.traj0 + (uint32_t)(r0 + ml);
    if (t < p.T && a < p.A) {
      const uint8_t* mask = p.mask + (p.step_mask ? (long)t * p.B * p.A : 0) + (long)(r0 + ml) * p.A;
      if (mask[a]) {
        const uint4 w = rng.block((uint32_t)a >> 2, step, traj, STREAM_CONTROLLER);
        cl.gum[o] = gumbel(word_to_uniform(word_of(w, a & 3)));
      }
    }
    if (p.use_done && t > 0) cl.ud[o] = word_to_uniform(rng.block(0, step - 1u, traj, STREAM_DONE).x);
  }
}

// LDS barrier that does not wait for the vector memory loads in flight
// (the gate phase's staging).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" : : : "memory");
}

// The owner's decisions for its rows at step t (t == T: only transition
// T-1 and the final done state).  All threads take part.
__device__ __forceinline__ void ctrl_owner(const PArgs& p, const CtrlLane& cl, char* lds, int t, int r0, int nrows) {
  const int tid = threadIdx.x, s = blockIdx.x >> 3, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int B = p.B, Z = p.Z, A = p.A;
  float* zrow = reinterpret_cast<float*>(lds + p.off_ctl);  // [Z]
  float* wbest = zrow + 160;                                // [4] best score per wave
  int* widx = reinterpret_cast<int*>(wbest + 4);             // [4] its action
  const rsrc_t rwc = make_rsrc(p.Wc, (uint32_t)(p.Nc * p.ldk * 4));
#pragma unroll
  for (int o = 0; o < kMaxOwn; ++o) {
    const int ml = s + kMembers * o;
    if (ml >= nrows) break;  // uniform
    const int m = r0 + ml;
    const rsrc_t rl = make_rsrc(p.Lh + (long)m * p.Nc, (uint32_t)(p.Nc * 4));
    float best = -INFINITY;
    int bi = -1;
    if (t < p.T) {
      // z_t of the row (written by mdn(t-1), or before the launch for t = 0)
      const rsrc_t rz = make_rsrc(p.z_out + ((long)t * B + m) * Z, (uint32_t)(Z * 4));
      if (tid < Z) zrow[tid] = __uint_as_float(cload4(rz, (uint32_t)tid * 4u));
      const float lh = __uint_as_float(cload4(rl, tid < A ? (uint32_t)tid * 4u : kOffNone));
      lds_barrier();
      if (tid < A && cl.gum[o] != -INFINITY) {
        float4 acc4 = make_float4(0.f, 0.f, 0.f, 0.f);
        const uint32_t wrow = (uint32_t)(tid * p.ldk) * 4u;
        for (int j = 0; j < Z; j += 4) {
          const float4 wv = as_float4(bload16(rwc, wrow + (uint32_t)j * 4u));
          const float4 zv = *reinterpret_cast<const float4*>(zrow + j);
          acc4.x = fmaf(wv.x, zv.x, acc4.x);
          acc4.y = fmaf(wv.y, zv.y, acc4.y);
          acc4.z = fmaf(wv.z, zv.z, acc4.z);
          acc4.w = fmaf(wv.w, zv.w, acc4.w);
        }
        best = (((acc4.x + acc4.y) + (acc4.z + acc4.w)) + lh) + cl.gum[o];
        bi = tid;
      }
      // best valid action, lowest index on ties
      wave_argmax(best, bi);
      if (lane == 0) {
        wbest[wave] = best;
        widx[wave] = bi;
      }
      lds_barrier();
    }
    if (tid == 0) {
      if (t < p.T) {  // thread 0 holds wave 0's best; the other waves'
        for (int w = 1; w < 4; ++w) {
          const float ob = wbest[w];
          const int oi = widx[w];
          if (oi >= 0 && (bi < 0 || ob > best || (ob == best && oi < bi))) {
            best = ob;
            bi = oi;
          }
        }
      }
      int* ds_l = row_done(p, lds);
      int* pv_l = row_prev(p, lds);
      int ds = ds_l[ml];
      if (pv_l[ml] >= 0) {  // transition t-1 was live: its reward and done
        const float rr = __uint_as_float(cload4(rl, (uint32_t)A * 4u));
        const float rd = __uint_as_float(cload4(rl, (uint32_t)(A + 1) * 4u));
        const int d = p.use_done ? sigmoidf(rd) > cl.ud[o] : 0;
        p.rewards[(long)(t - 1) * B + m] = rr;
        p.dones[(long)(t - 1) * B + m] = (uint8_t)d;
        if (d) ds = 1;
      }
      if (t < p.T) {
        const bool pad = t >= row_len(p, lds)[ml];
        int act = bi;
        if (ds || pad) act = -1;
        else if (act < 0) ds = 1;
        p.actions[(long)t * B + m] = act;
        if (act < 0) {
          p.rewards[(long)t * B + m] = 0.f;
          p.dones[(long)t * B + m] = pad ? 0 : 1;
        }
        pv_l[ml] = act;
        const rsrc_t rf = make_rsrc(p.flags + r0, (uint32_t)nrows * 4u);
        bstore4(rf, (uint32_t)ml * 4u, row_flag(t, act));
      } else {
        p.done_state[m] = ds;  // for the finishing kernel
      }
      ds_l[ml] = ds;
    }
  }
}

// The owner's decisions with one wave (A <= 64: lane a takes action a), so
// that the work-group's other three waves issue the gate phase's staging
// loads meanwhile and this wave's loads wait for nothing else.  Same
// arithmetic and tie rule as ctrl_owner.  Wave 0 only.
__device__ __forceinline__ void ctrl_owner_w0(const PArgs& p, const CtrlLane& cl, char* lds, int t, int r0,
                                              int nrows) {
  const int lane = threadIdx.x & 63, s = blockIdx.x >> 3;
  const int B = p.B, Z = p.Z, A = p.A;
  float* zrow = reinterpret_cast<float*>(lds + p.off_ctl);  // [Z]
  const rsrc_t rwc = make_rsrc(p.Wc, (uint32_t)(p.Nc * p.ldk * 4));
#pragma unroll
  for (int o = 0; o < kMaxOwn; ++o) {
    const int ml = s + kMembers * o;
    if (ml >= nrows) break;  // uniform
    const int m = r0 + ml;
    const rsrc_t rl = make_rsrc(p.Lh + (long)m * p.Nc, (uint32_t)(p.Nc * 4));
    // transition t-1's reward and done logits, loaded with the row's inputs
    const float rr = __uint_as_float(cload4(rl, (uint32_t)A * 4u));
    const float rd = __uint_as_float(cload4(rl, (uint32_t)(A + 1) * 4u));
    float best = -INFINITY;
    int bi = -1;
    if (t < p.T) {
      // z_t of the row (written by mdn(t-1), or before the launch for t = 0)
      const rsrc_t rz = make_rsrc(p.z_out + ((long)t * B + m) * Z, (uint32_t)(Z * 4));
      for (int j = lane; j < Z; j += 64) zrow[j] = __uint_as_float(cload4(rz, (uint32_t)j * 4u));
      const float lh = __uint_as_float(cload4(rl, lane < A ? (uint32_t)lane * 4u : kOffNone));
      // one wave: its LDS writes and reads are processed in order
      __builtin_amdgcn_wave_barrier();
      if (lane < A && cl.gum[o] != -INFINITY) {
        float4 acc4 = make_float4(0.f, 0.f, 0.f, 0.f);
        const uint32_t wrow = (uint32_t)(lane * p.ldk) * 4u;
        for (int j = 0; j < Z; j += 4) {
          const float4 wv = as_float4(bload16(rwc, wrow + (uint32_t)j * 4u));
          const float4 zv = *reinterpret_cast<const float4*>(zrow + j);
          acc4.x = fmaf(wv.x, zv.x, acc4.x);
          acc4.y = fmaf(wv.y, zv.y, acc4.y);
          acc4.z = fmaf(wv.z, zv.z, acc4.z);
          acc4.w = fmaf(wv.w, zv.w, acc4.w);
        }
        best = (((acc4.x + acc4.y) + (acc4.z + acc4.w)) + lh) + cl.gum[o];
        bi = lane;
      }
      // best valid action, lowest index on ties
      wave_argmax(best, bi);
      __builtin_amdgcn_wave_barrier();  // zrow is read out before the next row's z
    }
    if (lane == 0) {
      int* ds_l = row_done(p, lds);
      int* pv_l = row_prev(p, lds);
      int ds = ds_l[ml];
      if (pv_l[ml] >= 0) {  // transition t-1 was live: its reward and done
        const int d = p.use_done ? sigmoidf(rd) > cl.ud[o] : 0;
        p.rewards[(long)(t - 1) * B + m] = rr;
        p.dones[(long)(t - 1) * B + m] = (uint8_t)d;
        if (d) ds = 1;
      }
      if (t < p.T) {
        const bool pad = t >= row_len(p, lds)[ml];
        int act = bi;
        if (ds || pad) act = -1;
        else if (act < 0) ds = 1;
        p.actions[(long)t * B + m] = act;
        if (act < 0) {
          p.rewards[(long)t * B + m] = 0.f;
          p.dones[(long)t * B + m] = pad ? 0 : 1;
        }
        pv_l[ml] = act;
        const rsrc_t rf = make_rsrc(p.flags + r0, (uint32_t)nrows * 4u);
        bstore4(rf, (uint32_t)ml * 4u, row_flag(t, act));
      } else {
        p.done_state[m] = ds;  // for the finishing kernel
      }
      ds_l[ml] = ds;
    }
  }
}

// The actions of step t of all of the XCD's rows into LDS, once their owners'
// flags show them.  The wait is bounded: on timeout (or another work-group's)
// the error word is set and the work-group leaves at its next barrier.
__device__ __forceinline__ void ctrl_gather(const PArgs& p, char* lds, int t, int r0, int nrows, unsigned* err) {
  const int tid = threadIdx.x;
  if (tid < nrows) {
    const rsrc_t rf = make_rsrc(p.flags + r0, (uint32_t)nrows * 4u);
    unsigned spins = 0;
    uint32_t f = cload4(rf, (uint32_t)tid * 4u);
    while ((int)((f >> kFlagShift) - (uint32_t)(t + 1)) < 0) {
      if ((++spins & 63u) == 0) {
        if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
        if (spins >= kSpinLimit) {
          __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
      }
      __builtin_amdgcn_s_sleep(1);
      f = cload4(rf, (uint32_t)tid * 4u);
    }
    row_act(p, lds)[tid] = (int)(f & ((1u << kFlagShift) - 1u)) - 1;
  }
}

// ---------------------------------------------------------------------------
// gates(t): X_in -> h_{t+1} into X_out (rollout: with the step's actions)
// ---------------------------------------------------------------------------
template <int RB, int NBC, bool NLL>
__device__ __forceinline__ void gates_phase(const PArgs& p, GateState<RB, NBC>& st, const CtrlLane& cl,
                                            char* lds,
                                            int t, const float* Xin, float* Xout, int r0, int nrows) {
  constexpr int KSPLIT = GateState<RB, NBC>::KSPLIT;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, r16 = lane & 15;
  const int s = blockIdx.x >> 3;
  const int wb = wave % NBC, kp = wave / NBC;
  const int blk = s * NBC + wb;
  const int unit = 4 * blk + g;
  const bool owner = kp == 0;
  const int nks = (p.Z + p.H + 15) >> 4;  // K slices holding z, h (the padding columns are zero)
  const int nper = (nks + KSPLIT - 1) / KSPLIT;
  const int sl0 = kp * nper;
  const int B = p.B, H = p.H, A = p.A;

  // epilogue inputs issued first (older than the staging loads): the NLL
  // pass's actions
  int act[RB];
  if constexpr (NLL) {
    const rsrc_t ra = make_rsrc(p.actions + (long)t * B + r0, (uint32_t)nrows * 4u);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int ml = 16 * rb + r16;
      act[rb] = owner && ml < nrows ? (int)cload4(ra, (uint32_t)ml * 4u) : -1;
    }
  }

  // stage X_in rows [r0, r0 + nrows), columns [0, ldk) into LDS as
  // [slice][row block][16 rows][16 floats], in four chunks of local K slices.
  // Chunk c's LDS-DMA instructions, ordered (K part, slice, row block), are
  // dealt round-robin to the waves.  Chunk 0 goes out first; the loads of
  // chunk c+1 are then spread between the MFMAs of chunk c, so that the MFMA
  // pipe keeps running while they stream in.
  static_assert(KSPLIT <= 2, "one or two K parts per gate block");
  const u32x4 rsx = rsrc_words(Xin + (long)r0 * p.ldx, (uint32_t)(nrows * p.ldx * 4));
  const uint32_t lds0 = lds_addr(lds);
  const uint32_t ldxb = (uint32_t)p.ldx * 4u;
  const int rbv = (nrows + 15) >> 4;  // row blocks holding valid rows
  // A work-group that owns rows of a rollout with at most 64 actions makes
  // their decisions in wave 0 (ctrl_owner_w0) and deals the staging loads
  // to waves 1..3 only; every other work-group deals them to all four.
  const bool w0ctl = !NLL && p.A <= 64 && s < nrows;  // uniform
  const int nwi = w0ctl ? 3 : 4, wi = w0ctl ? wave - 1 : wave;
  auto valid_in = [&](int c, int kq) { return max(0, min(min(9, nper - 9 * c), nks - kq * nper - 9 * c)); };
  auto wave_count = [&](int c) {
    int n = valid_in(c, 0) * rbv;
    if (KSPLIT > 1) n += valid_in(c, 1) * rbv;
    return wi >= 0 && n > wi ? (n - wi + nwi - 1) / nwi : 0;
  };
  // the (slice, row block) of load k of chunk c of this wave
  auto piece = [&](int c, int k, int& sl, int& rb) {
    int r = wi + nwi * k, kq = 0;
    const int n0 = valid_in(c, 0) * rbv;
    if (KSPLIT > 1 && r >= n0) {
      kq = 1;
      r -= n0;
    }
    const int q = RB == 1 ? r : (rbv == RB ? r / RB : r / rbv);
    sl = kq * nper + 9 * c + q;
    rb = r - q * (RB == 1 ? 1 : rbv);
  };
  auto issue = [&](int c, int k) {
    int sl, rb;
    piece(c, k, sl, rb);
    const uint32_t voff = (uint32_t)(16 * rb + (lane >> 2)) * ldxb + (uint32_t)sl * 64u + (uint32_t)(lane & 3) * 16u;
    // The NLL recurrence keeps every X_t (no ring), so this CU has never
    // read these lines before and its L1 cannot hold a stale copy: the
    // plain policy suffices there (NLL recurrence 19.7 -> 19.3 us per step
    // at B = 512). The rollout reuses a two-matrix ring and needs the
    // device-coherent policy.
    if constexpr (NLL) dma16(rsx, voff, lds0 + (uint32_t)(sl * RB + rb) * 1024u);
    else cdma16(rsx, voff, lds0 + (uint32_t)(sl * RB + rb) * 1024u);
  };
  // few loads per wave (small batches): every chunk goes out at once and
  // one wait covers them all; else chunk 0 now and the rest under the MFMAs.
  // Decided for the whole work-group, so that the waves' barriers pair up:
  // at most 48 loads in all, so at most 12 per wave.
  int nall = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) nall += (valid_in(c, 0) + (KSPLIT > 1 ? valid_in(c, 1) : 0)) * rbv;
  const bool eager = nall <= 48;
  {
    const int n0 = wave_count(0);
    for (int k = 0; k < n0; ++k) issue(0, k);
    if (eager) {
      for (int c = 1; c < 4; ++c) {
        const int nc = wave_count(c);
        for (int k = 0; k < nc; ++k) issue(c, k);
      }
    }
  }
  // rollout: this work-group's rows' decisions, under the staging loads
  if constexpr (!NLL) {
    if (p.A <= 64) {
      if (w0ctl && wave == 0) ctrl_owner_w0(p, cl, lds, t, r0, nrows);
    } else {
      ctrl_owner(p, cl, lds, t, r0, nrows);
    }
  }

  // two accumulator sets (even and odd K slices) and RB row blocks give
  // 2 RB independent MFMA chains, issued interleaved
  f32x4 acc2[2][RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc2[0][rb] = acc2[1][rb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nval = min(nper, nks - sl0);  // this wave's valid K slices (uniform)
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    // with every chunk already in LDS (eager) a chunk past this wave's K
    // slices has nothing left to do; leaving here skips the scalar
    // bookkeeping of the remaining unrolled chunks (tiny rollout: about
    // 2.7k cycles per step)
    if (c > 0 && eager && 9 * c >= nval) break;
    if (c == 0 || !eager) {
      vm_wait<0>();  // this wave's loads of chunk c (the only ones in flight)
      __builtin_amdgcn_s_barrier();
      asm volatile("" : : : "memory");
    }
    const int nn = c < 3 && !eager ? wave_count(c + 1) : 0;
    int kk = 0;  // next load of chunk c+1 to issue
    const char* sb0 = lds + sl0 * RB * 1024 + 64 * r16 + 16 * g;
    if (9 * c + 9 <= nval && rbv == RB) {
      // whole chunk, every row block: straight-line MFMAs, slices in pairs;
      // the next pair's fragments are read from LDS before this pair's
      // MFMAs, so that their latency passes under them
      uint4 b0[RB], b1[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        b0[rb] = *reinterpret_cast<const uint4*>(sb0 + (9 * c * RB + rb) * 1024);
        b1[rb] = *reinterpret_cast<const uint4*>(sb0 + ((9 * c + 1) * RB + rb) * 1024);
      }
#pragma unroll
      for (int i = 9 * c; i < 9 * c + 9; i += 2) {
        const bool two = i + 1 < 9 * c + 9;
        const bool more = i + 2 < 9 * c + 9, more2 = i + 3 < 9 * c + 9;
        uint4 n0[RB], n1[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          if (more) n0[rb] = *reinterpret_cast<const uint4*>(sb0 + ((i + 2) * RB + rb) * 1024);
          if (more2) n1[rb] = *reinterpret_cast<const uint4*>(sb0 + ((i + 3) * RB + rb) * 1024);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            mfma4(acc2[i & 1][rb], st.wr[i], b0[rb], v);
            if (two) mfma4(acc2[(i + 1) & 1][rb], st.wr[i + 1], b1[rb], v);
          }
        const int upto = ((i - 9 * c + (two ? 2 : 1)) * nn + 8) / 9;
        for (; kk < upto; ++kk) issue(c + 1, kk);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          if (more) b0[rb] = n0[rb];
          if (more2) b1[rb] = n1[rb];
        }
      }
    } else {
#pragma unroll
      for (int i = 9 * c; i < 9 * c + 9; ++i) {
        if (i < nval) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            if (rb < rbv)
              Mfma<float>::step(acc2[i & 1][rb], st.wr[i], *reinterpret_cast<const uint4*>(sb0 + (i * RB + rb) * 1024));
        }
        const int upto = ((i - 9 * c + 1) * nn + 8) / 9;
        for (; kk < upto; ++kk) issue(c + 1, kk);
      }
    }
  }
  f32x4 acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = acc2[0][rb] + acc2[1][rb];

  // K-split partials meet in LDS (waves of the same gate block)
  f32x4* red = reinterpret_cast<f32x4*>(lds + p.off_red);
  if constexpr (KSPLIT > 1) {
    if (!owner) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) red[(((kp - 1) * NBC + wb) * RB + rb) * 64 + lane] = acc[rb];
    }
  }
  if constexpr (KSPLIT > 1 || !NLL) __syncthreads();
  if constexpr (KSPLIT > 1) {
    if (owner) {
#pragma unroll
      for (int k2 = 1; k2 < KSPLIT; ++k2)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc[rb] += red[(((k2 - 1) * NBC + wb) * RB + rb) * 64 + lane];
    }
  }
  if constexpr (!NLL) {
    // the rows' actions, from their owners
    if (wave == 0) ctrl_gather(p, lds, t, r0, nrows, sync_err(p));
    __syncthreads();
    const int* act_l = row_act(p, lds);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int ml = 16 * rb + r16;
      act[rb] = owner && ml < nrows ? act_l[ml] : -1;
    }
  }

  if (owner) {
    const rsrc_t rxo = make_rsrc(Xout + (long)r0 * p.ldx, (uint32_t)(nrows * p.ldx * 4));
    const rsrc_t rw = make_rsrc(p.WaT, (uint32_t)(A * 4 * H * 4));
    const bool tr = p.h_trace != nullptr, tc = p.c_trace != nullptr;
    const rsrc_t rht = make_rsrc(tr ? p.h_trace + ((long)(t + 1) * B + r0) * H : nullptr, tr ? (uint32_t)(nrows * H * 4) : 0u);
    const rsrc_t rct = make_rsrc(tc ? p.c_trace + ((long)(t + 1) * B + r0) * H : nullptr, tc ? (uint32_t)(nrows * H * 4) : 0u);
    const int hcol = p.Z + unit;  // X column of this lane's h
    const float* wat = reinterpret_cast<const float*>(lds + p.off_wat);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int ml = 16 * rb + r16;
      const bool ok = ml < nrows;
      const int a = act[rb];
      const bool live = NLL || a >= 0;
      const bool gather = ok && a >= 0 && a < A;
      float4 add;
      if (p.wat_lds) {
        add = gather ? *reinterpret_cast<const float4*>(wat + (a * NBC * 4 + 4 * wb + g) * 4)
                     : make_float4(0.f, 0.f, 0.f, 0.f);
      } else {
        add = as_float4(bload16(rw, gather ? (uint32_t)((a * 4 * H + 4 * unit) * 4) : kOffNone));
      }
      const float pi = acc[rb][0] + st.bias.x + add.x, pf = acc[rb][1] + st.bias.y + add.y;
      const float pg = acc[rb][2] + st.bias.z + add.z, po = acc[rb][3] + st.bias.w + add.w;
      const float gi = fsigmoid(pi), gf = fsigmoid(pf), gg = ftanh(pg), go = fsigmoid(po);
      float cn = gf * st.cst[rb] + gi * gg;
      float hn = go * ftanh(cn);
      if constexpr (NLL) {
        // the gate activations of row ml, unit `unit`, for the training
        // gradient (dropped without a trace)
        const bool tg = p.g_trace != nullptr;
        const rsrc_t rgt = make_rsrc(tg ? p.g_trace + ((long)t * B + r0) * 4 * H : nullptr,
                                     tg ? (uint32_t)(nrows * 4 * H * 4) : 0u);
        bstore16(rgt, ok ? (uint32_t)(ml * 4 * H + 4 * unit) * 4u : kOffNone,
                 make_uint4(__float_as_uint(gi), __float_as_uint(gf), __float_as_uint(gg), __float_as_uint(go)));
      }
      if (!live) {
        cn = st.cst[rb];
        hn = *reinterpret_cast<const float*>(lds + ((hcol >> 4) * RB + rb) * 1024 + 64 * r16 + 4 * (hcol & 15));
      }
      if (ok) st.cst[rb] = cn;
      const uint32_t ox = ok ? (uint32_t)ml * ldxb + (uint32_t)hcol * 4u : kOffNone;
      bstore4(rxo, ox, __float_as_uint(hn));
      const uint32_t oh = ok ? (uint32_t)(ml * H + unit) * 4u : kOffNone;
      bstore4(rht, oh, __float_as_uint(hn));  // dropped without traces
      bstore4(rct, oh, __float_as_uint(cn));
    }
  }
}

// ---------------------------------------------------------------------------
// mdn(t): mixture head on h_{t+1} (X_out columns Z ..), z_{t+1}, and the
// controller's h part of step t+1
// ---------------------------------------------------------------------------
// One tile: rows 16 rb .. 16 rb + 15 against HZ ? QC mixture blocks of dim
// group J (output rows 16 Q J ..) : none, plus HC ? controller block cb
// (W_c rows 16 cb .., h columns) : none; K (= H) split over the four waves,
// partial sums met in LDS.  QC (= p.Q) is compile-time: every guard on q is
// then resolved at compile time; under a runtime Q the guarded fragment
// loads keep the compiler from counting the loads in flight, and it waits
// for nearly all of them before each MFMA (medium rollout 23.5 against 21.9
// us per step).  `pre` is the lane's mixture noise drawn at the barrier
// (null: draw it here).
// MS: the K loop's slices per wave at most (kMaxMS, or fewer where the
// caller knows the call's H needs fewer)
template <int QC, bool HZ, bool HC, bool RES = false, int MS = kMaxMS>
__device__ __forceinline__ void mdn_tile(const PArgs& p, char* lds, int t, float* Xout, int r0, int nrows,
                                         int J, int rb, int cb, const MdnNoise* pre, const uint4* res = nullptr) {
  constexpr int NB = (HZ ? QC : 0) + (HC ? 1 : 0);  // A blocks of the tile
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, r16 = lane & 15;
  const int B = p.B, Z = p.Z, H = p.H;
  const int nsl = H >> 4;
  const int per = (nsl + 3) >> 2;  // K slices per wave (<= MS)
  const int s0 = wave * per;
  const uint32_t step = p.step0 + (uint32_t)t;
  const uint32_t ldxb = (uint32_t)p.ldx * 4u;
  const rsrc_t rwm = make_rsrc(p.Wm, (uint32_t)((16 * QC * (Z >> 2) + 16) * p.ldh * 4));
  const rsrc_t rwc = make_rsrc(p.Wc, (uint32_t)(p.Nc * p.ldk * 4));
  const rsrc_t rx = make_rsrc(Xout + (long)r0 * p.ldx, (uint32_t)(nrows * p.ldx * 4));
  const rsrc_t rzp = make_rsrc(p.z_out + ((long)t * B + r0) * Z, (uint32_t)(nrows * Z * 4));
  const rsrc_t rzn = make_rsrc(p.z_out + ((long)(t + 1) * B + r0) * Z, (uint32_t)(nrows * Z * 4));
  f32x4* red = reinterpret_cast<f32x4*>(lds + p.off_mdn);  // [4 waves][NB][64 lanes]

  const int ml = 16 * rb + r16, j = 4 * J + g;
  const bool ok = ml < nrows;
  // wave 0 owns the epilogue: liveness, noise or the frozen latent
  bool live = false;
  float zprev = 0.f;
  MdnNoise nz{};
  if (HZ && wave == 0) {
    live = ok && row_act(p, lds)[ml] >= 0;
    if (pre) nz = *pre;
    else if (live) nz = mixture_noise(Rng{p.k0, p.k1}, p.K, step, p.traj0 + (uint32_t)(r0 + ml), j);
    zprev = __uint_as_float(cload4(rzp, ok && !live ? (uint32_t)(ml * Z + j) * 4u : kOffNone));
  }
  // the epilogue's biases, fetched before the MFMAs
  float4 bz[HZ ? QC : 1], bcv = make_float4(0.f, 0.f, 0.f, 0.f);
  if (wave == 0) {
    if constexpr (HZ) {
#pragma unroll
      for (int q = 0; q < QC; ++q) bz[q] = *reinterpret_cast<const float4*>(p.bm + 16 * QC * J + 16 * q + 4 * g);
    }
    if constexpr (HC) bcv = *reinterpret_cast<const float4*>(p.bc + 16 * cb + 4 * g);
  }
  f32x4 acc[NB];
#pragma unroll
  for (int q = 0; q < NB; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  // slice i's fragments are fetched three slices ahead of their MFMAs; the
  // scheduling barriers keep the compiler from hoisting every fetch (which
  // would not fit the registers next to the resident gate weights)
  uint4 af[MS][NB], bf[MS];
#pragma unroll
  for (int i = 0; i < MS + 3; ++i) {
    if (i < MS) {
      const int sl = s0 + i;
      const bool kin = i < per && sl < nsl;
      const uint32_t kb = (uint32_t)(sl * 16 + 4 * g) * 4u;
      bf[i] = cload16(rx, kin && ok ? (uint32_t)ml * ldxb + (uint32_t)Z * 4u + kb : kOffNone);
#pragma unroll
      for (int q = 0; q < NB; ++q) {
        if constexpr (RES)
          af[i][q] = kin ? res[(sl * NB + q) * 64 + lane] : make_uint4(0u, 0u, 0u, 0u);
        else if (HZ && q < QC)
          af[i][q] = bload16(rwm, kin ? (uint32_t)((16 * QC * J + 16 * q + r16) * p.ldh) * 4u + kb : kOffNone);
        else
          af[i][q] = bload16(rwc, kin ? (uint32_t)((16 * cb + r16) * p.ldk + Z) * 4u + kb : kOffNone);
      }
    }
    if (i >= 3 && i - 3 < per && s0 + i - 3 < nsl) {
#pragma unroll
      for (int v = 0; v < 4; ++v)
#pragma unroll
        for (int q = 0; q < NB; ++q) mfma4(acc[q], af[i - 3][q], bf[i - 3], v);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int q = 0; q < NB; ++q) red[(wave * NB + q) * 64 + lane] = acc[q];
  __syncthreads();
  if (wave == 0 && ok) {
    if constexpr (HZ) {
      float z = zprev;
      if (live) {
        float feat[4 * QC];
#pragma unroll
        for (int q = 0; q < QC; ++q) {
          f32x4 v = red[q * 64 + lane] + red[(NB + q) * 64 + lane] + red[(2 * NB + q) * 64 + lane] +
                    red[(3 * NB + q) * 64 + lane];
          v += f32x4{bz[q].x, bz[q].y, bz[q].z, bz[q].w};
          feat[4 * q] = v[0]; feat[4 * q + 1] = v[1]; feat[4 * q + 2] = v[2]; feat[4 * q + 3] = v[3];
        }
        z = mixture_pick<QC>(p.K, p.tau, nz, feat, p.sig);
      }
      bstore4(rzn, (uint32_t)(ml * Z + j) * 4u, __float_as_uint(z));
      bstore4(rx, (uint32_t)ml * ldxb + (uint32_t)j * 4u, __float_as_uint(z));
    }
    if constexpr (HC) {
      constexpr int q = NB - 1;
      f32x4 v = red[q * 64 + lane] + red[(NB + q) * 64 + lane] + red[(2 * NB + q) * 64 + lane] +
                red[(3 * NB + q) * 64 + lane];
      v += f32x4{bcv.x, bcv.y, bcv.z, bcv.w};
      const rsrc_t rl = make_rsrc(p.Lh + (long)r0 * p.Nc, (uint32_t)(nrows * p.Nc * 4));
      bstore16(rl, (uint32_t)(ml * p.Nc + 16 * cb + 4 * g) * 4u,
               make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])));
    }
  }
  __syncthreads();
}

// Work-group s's single mdn tile, its weight fragments resident in LDS.
template <int QC, int MS>
__device__ __forceinline__ void mdn_phase_res(const PArgs& p, char* lds, int t, float* Xout, int r0, int nrows,
                                              const MdnNoise& pre, const uint4* res, int zt, int nt, int rbv) {
  const int s = blockIdx.x >> 3;
  if (s < zt) {
    const int J = s / rbv, rb = s % rbv;
    if (!p.ctl_sep && J < p.ncb) mdn_tile<QC, true, true, true, MS>(p, lds, t, Xout, r0, nrows, J, rb, J, &pre, res);
    else mdn_tile<QC, true, false, true, MS>(p, lds, t, Xout, r0, nrows, J, rb, 0, &pre, res);
  } else if (s < nt) {
    const int c = s - zt;
    mdn_tile<QC, false, true, true, MS>(p, lds, t, Xout, r0, nrows, 0, c / p.ncb, c % p.ncb, nullptr, res);
  }
}

// The tiles of one XCD: ZT = (Z/4) rbv mixture tiles, then (ctl_sep) the
// ncb rbv controller tiles; without ctl_sep the mixture tiles of dim groups
// J < ncb carry controller block J.  Work-group s takes tiles s, s + 32, ...
// `pre` holds the noise of tile s when it is a mixture tile.
template <int QC>
__device__ __forceinline__ void mdn_phase(const PArgs& p, char* lds, int t, float* Xout, int r0, int nrows,
                                          const MdnNoise& pre) {
  const int s = blockIdx.x >> 3;
  const int rbv = (nrows + 15) >> 4;
  const int zt = (p.Z >> 2) * rbv;
  const int nt = zt + (p.ctl_sep ? p.ncb * rbv : 0);
  if (p.mres) {
    // at most one tile per work-group, its weight fragments in LDS; with
    // H <= 256 the K loop is instantiated for its four slices per wave, so
    // that no iteration is spent on slices the call does not have
    const uint4* res = reinterpret_cast<const uint4*>(lds + p.off_mres);
    if (((p.H >> 4) + 3) >> 2 <= 4) mdn_phase_res<QC, 4>(p, lds, t, Xout, r0, nrows, pre, res, zt, nt, rbv);
    else mdn_phase_res<QC, kMaxMS>(p, lds, t, Xout, r0, nrows, pre, res, zt, nt, rbv);
    return;
  }
  for (int ti = s; ti < nt; ti += kMembers) {
    const MdnNoise* pn = ti == s ? &pre : nullptr;
    if (ti < zt) {
      const int J = ti / rbv, rb = ti % rbv;
      if (!p.ctl_sep && J < p.ncb) mdn_tile<QC, true, true>(p, lds, t, Xout, r0, nrows, J, rb, J, pn);
      else mdn_tile<QC, true, false>(p, lds, t, Xout, r0, nrows, J, rb, 0, pn);
    } else {
      const int c = ti - zt;
      mdn_tile<QC, false, true>(p, lds, t, Xout, r0, nrows, 0, c / p.ncb, c % p.ncb, nullptr);
    }
  }
}

// The controller tiles alone, over h_0 (X_0): Lh of step 0.
template <int QC>
__device__ __forceinline__ void ctrl_h0(const PArgs& p, char* lds, float* X0, int r0, int nrows) {
  const int s = blockIdx.x >> 3;
  const int rbv = (nrows + 15) >> 4;
  for (int c = s; c < p.ncb * rbv; c += kMembers)
    mdn_tile<QC, false, true>(p, lds, 0, X0, r0, nrows, 0, c / p.ncb, c % p.ncb, nullptr);
}

// The mixture noise of tile s of mdn(t) (wave 0's lanes), drawn at the
// barrier before it.
__device__ __forceinline__ void mdn_noise_pre(const PArgs& p, MdnNoise& nz, int t, int r0, int nrows) {
  const int s = blockIdx.x >> 3, lane = threadIdx.x & 63;
  const int rbv = (nrows + 15) >> 4;
  if ((threadIdx.x >> 6) != 0 || s >= (p.Z >> 2) * rbv) return;
  const int J = s / rbv, rb = s % rbv;
  const int ml = 16 * rb + (lane & 15), j = 4 * J + (lane >> 4);
  if (ml < nrows)
    nz = mixture_noise(Rng{p.k0, p.k1}, p.K, p.step0 + (uint32_t)t, p.traj0 + (uint32_t)(r0 + ml), j);
}

// ---------------------------------------------------------------------------
// The kernel.
// ---------------------------------------------------------------------------
// The kernel's arguments read again from the kernel-argument segment through
// a pointer the compiler cannot see through: values derived from them
// (buffer resources, offsets) are then recomputed in each phase instead of
// being kept across the step loop in scalar registers, which spilled.
__device__ __forceinline__ const PArgs& fresh_args() {
  auto a = (const __attribute__((address_space(4))) PArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(a));
  return *(const PArgs*)a;
}

template <int RB, int NBC, bool NLL, int QC>
__global__ void __launch_bounds__(256, 1) k_persist(const PArgs p) {
  // no static LDS: the dynamic region starts at LDS address 0, so that the
  // 1 KB LDS-DMA destinations are 1 KB aligned (misaligned ones run several
  // times slower); the two flags live in the last 64 bytes of the region
  extern __shared__ __attribute__((aligned(1024))) char lds[];
  int& s_flag = *reinterpret_cast<int*>(lds + p.off_flags);
  int& s_agent = *reinterpret_cast<int*>(lds + p.off_flags + 4);
  constexpr int KSPLIT = 4 / NBC;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, g = lane >> 4, r16 = lane & 15;
  const int x = blockIdx.x & 7, s = blockIdx.x >> 3;
  const int r0 = x * p.Bx;
  const int nrows = min(p.Bx, p.B - r0);
  if (nrows <= 0) return;  // the whole group leaves

  GroupSync gs{sync_ctr(p, x), sync_err(p), 0u, false,
               p.stamps && tid == 0 ? p.stamps + (long)blockIdx.x * p.nst : nullptr, p.nst};
  phase_stamp(gs.st, gs.nst, 0);
  // placement check, settled by the first barrier
  if (tid == 0 && xcc_id() != (unsigned)x)
    __hip_atomic_fetch_or(sync_flag(p, x), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // register-resident weights and state
  GateState<RB, NBC> st;
  const int wb = wave % NBC, kp = wave / NBC;
  const int blk = s * NBC + wb;
  const int unit = 4 * blk + g;
  const bool owner = kp == 0;
  const int nks = (p.Z + p.H + 15) >> 4;  // K slices holding z, h (the padding columns are zero)
  const int nper = (nks + KSPLIT - 1) / KSPLIT;
  const int sl0 = kp * nper;
  {
    const rsrc_t rwg = make_rsrc(p.Wg, (uint32_t)(4 * p.H * p.ldk * 4));
    const uint32_t rowb = (uint32_t)((16 * blk + r16) * p.ldk) * 4u;
#pragma unroll
    for (int i = 0; i < kMaxS; ++i) {
      const bool ok = i < nper && sl0 + i < nks;
      st.wr[i] = bload16(rwg, ok ? rowb + (uint32_t)((sl0 + i) * 16 + 4 * g) * 4u : kOffNone);
    }
    const rsrc_t rb4 = make_rsrc(p.bg, (uint32_t)(16 * p.H));
    st.bias = as_float4(bload16(rb4, owner ? (uint32_t)unit * 16u : kOffNone));
    const rsrc_t rc = make_rsrc(p.c + (long)r0 * p.H, (uint32_t)(nrows * p.H * 4));
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int ml = 16 * rb + r16;
      st.cst[rb] = __uint_as_float(bload4(rc, owner && ml < nrows ? (uint32_t)(ml * p.H + unit) * 4u : kOffNone));
    }
  }
  if constexpr (!NLL) {
    // row state: the actions of step t, the done state, the previous action
    int* rows = row_act(p, lds);
    for (int i = tid; i < 4 * 64; i += 256) {
      const int ml = i & 63;
      int v = -1;
      if (i >= 64 && i < 128) v = ml < nrows ? p.done_state[r0 + ml] : 0;
      if (i >= 192) v = p.lengths && ml < nrows ? p.lengths[r0 + ml] : 0x7fffffff;
      rows[i] = v;
    }
    // the flags of this work-group's rows start at 0 (before barrier 1)
#pragma unroll
    for (int o = 0; o < kMaxOwn; ++o) {
      const int ml = s + kMembers * o;
      if (tid == 0 && ml < nrows) p.flags[r0 + ml] = 0u;
    }
  }
  if constexpr (!NLL) {
    if (p.mres) {
      // the weight fragments of this work-group's mdn tile (the same for
      // every step), laid out as mdn_tile reads them
      const int rbv = (nrows + 15) >> 4, zt = (p.Z >> 2) * rbv;
      const int nt = zt + (p.ctl_sep ? p.ncb * rbv : 0);
      if (s < nt) {
        const bool hz = s < zt;
        const int J = hz ? s / rbv : 0;
        const bool hc = hz ? (!p.ctl_sep && J < p.ncb) : true;
        const int cb = hz ? J : (s - zt) % p.ncb;
        const int nb = (hz ? p.Q : 0) + (hc ? 1 : 0);
        uint4* res = reinterpret_cast<uint4*>(lds + p.off_mres);
        for (int idx = tid; idx < (p.H >> 4) * nb * 64; idx += 256) {
          const int ln = idx & 63, q = (idx >> 6) % nb, sl = (idx >> 6) / nb;
          const int kcol = sl * 16 + 4 * (ln >> 4);
          const float* src = hz && q < p.Q ? p.Wm + (long)(16 * p.Q * J + 16 * q + (ln & 15)) * p.ldh + kcol
                                           : p.Wc + (long)(16 * cb + (ln & 15)) * p.ldk + p.Z + kcol;
          res[idx] = *reinterpret_cast<const uint4*>(src);
        }
      }
    }
  }
  if (p.wat_lds) {
    // this work-group's columns of the one-hot block: [A][NBC blocks][4 units][4 gates]
    float* wat = reinterpret_cast<float*>(lds + p.off_wat);
    const int per_a = 16 * NBC;
    for (int i = tid; i < p.A * per_a; i += 256) {
      const int aa = i / per_a, r = i % per_a;
      wat[i] = p.WaT[(long)aa * 4 * p.H + 16 * NBC * s + r];
    }
  }

  if (!group_sync(gs, &s_flag)) return;
  if (tid == 0) s_agent = __hip_atomic_load(sync_flag(p, x), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
  __syncthreads();
  gs.agent = s_agent != 0;

  CtrlLane cl;
  MdnNoise nz{};
  if constexpr (!NLL) {
    // the h part of the step-0 controller logits, from h_0 (X_0, written
    // before the launch), like every later step's from mdn(t-1)
    ctrl_h0<QC>(p, lds, p.X, r0, nrows);
    group_arrive(gs);
    ctrl_noise(p, cl, 0, r0, nrows);
    if (!group_wait(gs, &s_flag)) return;
  }

  const long BX = (long)p.B * p.ldx;
  if constexpr (NLL) {
    for (int t = 0; t < p.T; ++t) {
      const PArgs& q = fresh_args();
      gates_phase<RB, NBC, true>(q, st, cl, lds, t, q.X + (long)t * BX, q.X + (long)(t + 1) * BX, r0, nrows);
      if (t + 1 < p.T && !group_sync(gs, &s_flag)) return;
    }
    __syncthreads();
    phase_stamp(gs.st, gs.nst, gs.nst - 1);
  } else {
    for (int t = 0; t < p.T; ++t) {
      const PArgs& q = fresh_args();
      float* Xt = q.X + (long)(t & 1) * BX;
      float* Xn = q.X + (long)((t + 1) & 1) * BX;
      gates_phase<RB, NBC, false>(q, st, cl, lds, t, Xt, Xn, r0, nrows);
      group_arrive(gs);
      mdn_noise_pre(fresh_args(), nz, t, r0, nrows);
      if (!group_wait(gs, &s_flag)) return;
      mdn_phase<QC>(fresh_args(), lds, t, Xn, r0, nrows, nz);
      group_arrive(gs);
      if (t + 1 < p.T) ctrl_noise(fresh_args(), cl, t + 1, r0, nrows);
      if (!group_wait(gs, &s_flag)) return;
    }
    // transition T-1 (its reward and done from mdn(T-1)'s Lh), the done state
    {
      const PArgs& q = fresh_args();
      ctrl_noise(q, cl, q.T, r0, nrows);
      if (q.A <= 64) {
        if ((threadIdx.x >> 6) == 0) ctrl_owner_w0(q, cl, lds, q.T, r0, nrows);
      } else {
        ctrl_owner(q, cl, lds, q.T, r0, nrows);
      }
    }
    // final cell state for k_rollout_finish
    if (owner) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int ml = 16 * rb + r16;
        if (ml < nrows) p.c[(long)(r0 + ml) * p.H + unit] = st.cst[rb];
      }
    }
    __syncthreads();
    phase_stamp(gs.st, gs.nst, gs.nst - 1);
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
constexpr size_t kLdsMax = 160 * 1024 - 64;  // LDS budget below the flags
constexpr size_t kLdsMin = 81 * 1024;        // above half the CU's LDS: one work-group per CU

bool persist_enabled() {
  const char* e = std::getenv("WM_PERSISTENT");
  return !(e && e[0] == '0');
}

// Row blocks per XCD for B rows (0 = not served by the persistent kernels).
int persist_rb(int B) {
  const int bx = (B + kGroups - 1) / kGroups;
  return bx <= 16 ? 1 : bx <= 32 ? 2 : bx <= 64 ? 4 : 0;
}

struct PPlan {
  int rb = 0, nbc = 0;
  size_t lds = 0;
  int off_red = 0, off_rows = 0, off_wat = 0, off_mdn = 0, off_ctl = 0, off_flags = 0, off_mres = 0;
  int wat_lds = 0, mres = 0;
  int ncb = 0, ctl_sep = 0;
};

// The grid must be co-resident with one work-group per CU: 8 XCDs x 32 CUs.
bool device_fits() {
  static int cached[64];  // 0 unknown, 1 fits, 2 does not
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return false;
  if (cached[dev] == 0) {
    int cus = 0;
    const bool ok = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
                    cus == kGrid;
    cached[dev] = ok ? 1 : 2;
  }
  return cached[dev] == 1;
}

bool plan(const Layout& L, int B, bool nll, PPlan& pl) {
  if (L.dt != 0) return false;
  if (L.H != 256 && L.H != 512) return false;
  if (L.Nc > 128 || L.K > 8) return false;
  const int rb = persist_rb(B);
  if (rb == 0) return false;
  const int nbc = L.H / 128;
  const int nks = (L.Z + L.H + 15) / 16;
  const int nper = (nks + 4 / nbc - 1) / (4 / nbc);
  if (nper > kMaxS || (L.H / 16 + 3) / 4 > kMaxMS || L.Q > kMaxQ) return false;
  if (L.N > 0) return false;  // the two-level controller runs on the multi-launch path
  pl.rb = rb;
  pl.nbc = nbc;
  if (!nll) {
    // the tiles of mdn(t): the controller's h-part blocks as tiles of their
    // own when all tiles fit one round of the 32 work-groups, else inside
    // the first mixture tiles; one thread per action in the owner decisions
    const int rbv = (((B + kGroups - 1) / kGroups) + 15) / 16;
    pl.ncb = L.Nc / 16;
    const int zt = (L.Z / 4) * rbv;
    pl.ctl_sep = zt + pl.ncb * rbv <= kMembers ? 1 : 0;
    if (!pl.ctl_sep && pl.ncb > L.Z / 4) return false;
    if (L.Z > 160 || L.A > 256) return false;
  }
  // the mixture-head partial sums share the gate staging's bytes (another
  // phase); the controller's scratch, the row state and the one-hot columns
  // persist
  size_t o = (size_t)nks * rb * 1024;  // staging
  pl.off_red = (int)o;
  o += (size_t)(4 - nbc) * rb * 1024;   // K-split partial sums
  pl.off_mdn = 0;
  if (!nll) {
    o = o > (size_t)4 * (L.Q + 1) * 1024 ? o : (size_t)4 * (L.Q + 1) * 1024;
    pl.off_ctl = (int)o;
    o += 1024;                        // a row's z_t, wave bests
    pl.off_rows = (int)o;
    o += (size_t)4 * 64 * 4;          // actions, done state, previous actions, horizons
  }
  o = (o + 15) & ~(size_t)15;
  pl.off_wat = (int)o;
  const size_t wat = (size_t)L.A * 64 * nbc;
  if (o + wat <= kLdsMax) {
    pl.wat_lds = 1;
    o += wat;
  }
  if (!nll) {
    // with at most one mdn tile per work-group, its weight fragments stay in
    // LDS for the whole call: [K slice][block][64 lanes] 16-byte pieces
    const int rbv = (((B + kGroups - 1) / kGroups) + 15) / 16;
    const int nt = (L.Z / 4) * rbv + (pl.ctl_sep ? pl.ncb * rbv : 0);
    const size_t res = (size_t)(L.H / 16) * (L.Q + 1) * 1024;
    if (nt <= kMembers && o + res <= kLdsMax) {
      pl.off_mres = (int)o;
      pl.mres = 1;
      o += res;
    }
  }
  if (o > kLdsMax) return false;
  o = o < kLdsMin ? kLdsMin : o;
  pl.off_flags = (int)((o + 15) & ~(size_t)15);
  pl.lds = (size_t)pl.off_flags + 64;
  return true;
}

template <int RB, int NBC, bool NLL, int QC>
hipError_t launch_k(const PArgs& a, size_t lds, hipStream_t s) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_persist<RB, NBC, NLL, QC>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  return launch(NLL ? "nll_persist" : "persist", k_persist<RB, NBC, NLL, QC>, dim3(kGrid), dim3(256), lds, s, a);
}

// the mixture head with its block count Q = ceil(3K / 4) (1 .. 6 for
// K <= 8) at compile time; the NLL recurrence has no mixture phase
template <int RB, int NBC, bool NLL>
hipError_t launch_q(const PArgs& a, size_t lds, hipStream_t s) {
  if constexpr (NLL) {
    return launch_k<RB, NBC, true, 0>(a, lds, s);
  } else {
    switch (a.Q) {
      case 1: return launch_k<RB, NBC, false, 1>(a, lds, s);
      case 2: return launch_k<RB, NBC, false, 2>(a, lds, s);
      case 3: return launch_k<RB, NBC, false, 3>(a, lds, s);
      case 4: return launch_k<RB, NBC, false, 4>(a, lds, s);
      case 5: return launch_k<RB, NBC, false, 5>(a, lds, s);
      case 6: return launch_k<RB, NBC, false, 6>(a, lds, s);
      default: return hipErrorNotSupported;
    }
  }
}

template <bool NLL>
hipError_t launch_plan(const PArgs& a, const PPlan& pl, hipStream_t s) {
  switch (pl.rb * 8 + pl.nbc) {
    case 1 * 8 + 2: return launch_q<1, 2, NLL>(a, pl.lds, s);
    case 1 * 8 + 4: return launch_q<1, 4, NLL>(a, pl.lds, s);
    case 2 * 8 + 2: return launch_q<2, 2, NLL>(a, pl.lds, s);
    case 2 * 8 + 4: return launch_q<2, 4, NLL>(a, pl.lds, s);
    case 4 * 8 + 2: return launch_q<4, 2, NLL>(a, pl.lds, s);
    case 4 * 8 + 4: return launch_q<4, 4, NLL>(a, pl.lds, s);
    default: return hipErrorNotSupported;
  }
}

PArgs base_args(const Packed& P, const PPlan& pl, int B, int T) {
  const Layout& L = P.L;
  const char* base = reinterpret_cast<const char*>(P.base);
  PArgs a{};
  a.Wg = reinterpret_cast<const float*>(base + L.off_Wg);
  a.WaT = reinterpret_cast<const float*>(base + L.off_WaT);
  a.bg = reinterpret_cast<const float*>(base + L.off_bg);
  a.Wm = reinterpret_cast<const float*>(base + L.off_Wm);
  a.bm = reinterpret_cast<const float*>(base + L.off_bm);
  a.Wc = reinterpret_cast<const float*>(base + L.off_Wc);
  a.bc = reinterpret_cast<const float*>(base + L.off_bc);
  a.Z = L.Z; a.H = L.H; a.A = L.A; a.K = L.K; a.Q = L.Q; a.Nc = L.Nc;
  a.ldk = L.ldk; a.ldh = L.ldh; a.ldx = L.ldx;
  a.B = B; a.T = T; a.Bx = (B + kGroups - 1) / kGroups;
  a.wat_lds = pl.wat_lds;
  a.mres = pl.mres;
  a.off_mres = pl.off_mres;
  a.off_red = pl.off_red; a.off_rows = pl.off_rows; a.off_wat = pl.off_wat;
  a.off_mdn = pl.off_mdn; a.off_ctl = pl.off_ctl; a.off_flags = pl.off_flags;
  a.ncb = pl.ncb;
  a.ctl_sep = pl.ctl_sep;
  return a;
}

}  // namespace

size_t persist_partial_bytes(const Layout& L, int B) {
  PPlan pl;
  if (!plan(L, B, false, pl)) return 0;
  return (size_t)B * L.Nc * 4 + (size_t)B * 4;  // Lh, then the row flags
}

bool persist_usable(const Layout& L, int B, bool nll) {
  PPlan pl;
  return persist_enabled() && plan(L, B, nll, pl) && device_fits();
}

// Phase stamps for a launch with `nbar` barriers, when phase timing is on.
void attach_stamps(PArgs& a, int nbar, bool nll, hipStream_t s) {
  const int nst = 2 * nbar + 2;
  a.stamps = phase_buffer((size_t)kGrid * nst, s);
  a.nst = a.stamps ? nst : 0;
  if (a.stamps) phase_layout(kGrid, nst, a.T, nll);
}

hipError_t launch_rollout_persist(const Packed& P, const RolloutBufs& R, hipStream_t s) {
  PPlan pl;
  if (!persist_enabled() || !plan(P.L, R.B, false, pl) || !R.P || !R.sync || !device_fits())
    return hipErrorNotSupported;
  PArgs a = base_args(P, pl, R.B, R.T);
  attach_stamps(a, 2 + 2 * R.T, false, s);
  a.k0 = R.k0; a.k1 = R.k1; a.traj0 = R.traj0; a.step0 = R.step0;
  a.tau = R.tau;
  a.sig = (R.flags & WM_FLAG_SIGMA_TAU) ? sqrtf(R.tau) : 1.0f;
  a.step_mask = (R.flags & WM_FLAG_STEP_MASK) != 0;
  a.use_done = (R.flags & WM_FLAG_DONE) != 0;
  a.X = reinterpret_cast<float*>(R.x);
  a.c = R.c;
  a.done_state = R.done_state;
  a.lengths = R.lengths;
  a.Lh = R.P;
  a.flags = reinterpret_cast<unsigned*>(R.P + (size_t)R.B * P.L.Nc);
  a.sync = R.sync;
  a.mask = R.mask;
  a.z_out = R.z_out;
  a.actions = R.actions;
  a.rewards = R.rewards;
  a.dones = R.dones;
  const bool trace = (R.flags & WM_FLAG_TRACE) != 0;
  a.h_trace = trace ? R.h_trace : nullptr;
  a.c_trace = trace ? R.c_trace : nullptr;
  return launch_plan<false>(a, pl, s);
}

hipError_t launch_nll_persist(const Packed& P, const NllBufs& N, hipStream_t s) {
  PPlan pl;
  if (!persist_enabled() || !plan(P.L, N.B, true, pl) || !N.sync || !device_fits())
    return hipErrorNotSupported;
  PArgs a = base_args(P, pl, N.B, N.T);
  attach_stamps(a, N.T, true, s);
  a.X = reinterpret_cast<float*>(N.x);
  a.c = N.c;
  a.sync = N.sync;
  a.actions = const_cast<int32_t*>(N.actions);
  a.g_trace = N.g_trace;
  a.c_trace = N.c_trace;
  return launch_plan<true>(a, pl, s);
}

}  // namespace wm
