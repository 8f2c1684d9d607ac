// HIP kernels of libwm for gfx950 (MI355X).
//
// The dream rollout runs three kernels per step, each a GEMM on the MFMA
// units with the step's arithmetic fused into its epilogue:
//   k_ctrl   controller logits W_c [z_t, h_t] (+ reward/done rows on h_t),
//            masked Gumbel-max action, resolution of the previous
//            transition's reward and done flag;
//   k_gates  gate GEMM [z_t, h_t] x W^T plus the gathered one-hot column,
//            LSTM cell, state commit (frozen rows copy their state);
//   k_mdn    mixture head on h_{t+1}, Gumbel-max component pick per latent
//            dim, Box-Muller draw, z_{t+1} commit.
// The activations of step t are one matrix X_t = [q(z_t) | h_t | 0] in the
// compute type (q: round to the compute type), so every GEMM streams a
// single K-contiguous operand: the gate and controller GEMMs read X_t from
// column 0, the mixture head reads X_{t+1} from column Z, k_gates writes h_{t+1}
// and k_mdn q(z_{t+1}) into X_{t+1}.
// The NLL pass runs k_gates once per step (teacher-forced), then one k_mdn
// over all T*B rows with a log-likelihood epilogue, then a deterministic
// reduction.  Nothing here allocates memory.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "wm_device.h"
#include "wm_kernels.h"
#include "wm_profile.h"

namespace wm {

static constexpr float kHalfLn2Pi = 0.91893853320467274178f;

// ===========================================================================
// Packing (one-time): canonical fp32 -> kernel layout, rounded to DT.
// ===========================================================================
template <typename DT>
__global__ void k_pack(const Layout L, char* base, const float* __restrict__ W_g,
                       const float* __restrict__ b_g, const float* __restrict__ W_m,
                       const float* __restrict__ b_m, const float* __restrict__ w_r,
                       const float* __restrict__ b_r, const float* __restrict__ w_d,
                       const float* __restrict__ b_d, const float* __restrict__ W_c,
                       const float* __restrict__ b_c) {
  const int Z = L.Z, H = L.H, A = L.A, K = L.K, Q = L.Q;
  const long cg = Z + A + H;  // canonical W_g row length
  const int section = blockIdx.y;
  const long stride = (long)gridDim.x * blockDim.x;
  const long i0 = (long)blockIdx.x * blockDim.x + threadIdx.x;
  DT* Wg = reinterpret_cast<DT*>(base + L.off_Wg);
  DT* WaT = reinterpret_cast<DT*>(base + L.off_WaT);
  float* bg = reinterpret_cast<float*>(base + L.off_bg);
  DT* Wm = reinterpret_cast<DT*>(base + L.off_Wm);
  float* bm = reinterpret_cast<float*>(base + L.off_bm);
  DT* Wc = reinterpret_cast<DT*>(base + L.off_Wc);
  float* bc = reinterpret_cast<float*>(base + L.off_bc);
  const int head0 = 16 * Q * (Z / 4);
  if (section == 0) {
    for (long idx = i0; idx < (long)4 * H * L.ldk; idx += stride) {
      const int r = (int)(idx / L.ldk), col = (int)(idx % L.ldk);
      const long crow = (long)(r % 4) * H + r / 4;
      float v = 0.f;
      if (col < Z) v = W_g[crow * cg + col];
      else if (col < Z + H) v = W_g[crow * cg + A + col];
      DType<DT>::store(Wg, idx, v);
    }
  } else if (section == 1) {
    for (long idx = i0; idx < (long)A * 4 * H; idx += stride) {
      const int a = (int)(idx / (4 * H)), r = (int)(idx % (4 * H));
      const long crow = (long)(r % 4) * H + r / 4;
      DType<DT>::store(WaT, idx, W_g[crow * cg + Z + a]);
    }
  } else if (section == 2) {
    for (long idx = i0; idx < 4 * H; idx += stride) bg[idx] = b_g[(idx % 4) * H + idx / 4];
  } else if (section == 3 || section == 4) {
    const long n = section == 3 ? (long)L.Nm * L.ldh : (long)L.Nm;
    for (long idx = i0; idx < n; idx += stride) {
      const int row = section == 3 ? (int)(idx / L.ldh) : (int)idx;
      const int col = section == 3 ? (int)(idx % L.ldh) : 0;
      float v = 0.f;
      if (col < H) {
        if (row >= head0) {
          const int hr = row - head0;
          if (section == 3) v = hr == 0 ? w_r[col] : (hr == 1 ? w_d[col] : 0.f);
          else v = hr == 0 ? b_r[0] : (hr == 1 ? b_d[0] : 0.f);
        } else {
          const int J = row / (16 * Q), rem = row % (16 * Q);
          const int q = rem / 16, g = (rem % 16) / 4, vv = rem % 4;
          const int j = 4 * J + g, f = 4 * q + vv;
          long canon = -1;
          if (f < K) canon = (long)j * K + f;
          else if (f < 2 * K) canon = (long)Z * K + (long)j * K + (f - K);
          else if (f < 3 * K) canon = 2L * Z * K + (long)j * K + (f - 2 * K);
          if (canon >= 0) v = section == 3 ? W_m[canon * H + col] : b_m[canon];
        }
      }
      if (section == 3) DType<DT>::store(Wm, idx, v);
      else bm[idx] = v;
    }
  } else if (section == 5) {
    for (long idx = i0; idx < (long)L.Nc * L.ldk; idx += stride) {
      const int row = (int)(idx / L.ldk), col = (int)(idx % L.ldk);
      float v = 0.f;
      if (col < Z + H) {
        const int Ac = L.Ac;
        if (row < Ac) v = W_c[(long)row * (Z + H) + col];
        else if (row == Ac && col >= Z) v = w_r[col - Z];
        else if (row == Ac + 1 && col >= Z) v = w_d[col - Z];
      }
      DType<DT>::store(Wc, idx, v);
    }
  } else if (section == 6) {
    for (long idx = i0; idx < L.Nc; idx += stride)
      bc[idx] = idx < L.Ac ? b_c[idx] : (idx == L.Ac ? b_r[0] : (idx == L.Ac + 1 ? b_d[0] : 0.f));
  } else if constexpr (sizeof(DT) == 4) {
    if (section == 7) {  // WhT[i][r] = Wg[r][Z + i]
      float* WhT = reinterpret_cast<float*>(base + L.off_WhT);
      for (long idx = i0; idx < (long)H * 4 * H; idx += stride) {
        const int i = (int)(idx / (4 * H)), r = (int)(idx % (4 * H));
        WhT[idx] = W_g[((long)(r % 4) * H + r / 4) * cg + A + Z + i];
      }
    } else if (section == 8) {  // WmT[i][r] = Wm[r][i], zero past Nm
      float* WmT = reinterpret_cast<float*>(base + L.off_WmT);
      for (long idx = i0; idx < (long)H * L.NmP; idx += stride) {
        const int i = (int)(idx / L.NmP), row = (int)(idx % L.NmP);
        float v = 0.f;
        if (row >= head0 && row < L.Nm) {
          const int hr = row - head0;
          v = hr == 0 ? w_r[i] : (hr == 1 ? w_d[i] : 0.f);
        } else if (row < head0) {
          const int J = row / (16 * Q), rem = row % (16 * Q);
          const int q = rem / 16, g = (rem % 16) / 4, vv = rem % 4;
          const int j = 4 * J + g, f = 4 * q + vv;
          long canon = -1;
          if (f < K) canon = (long)j * K + f;
          else if (f < 2 * K) canon = (long)Z * K + (long)j * K + (f - K);
          else if (f < 3 * K) canon = 2L * Z * K + (long)j * K + (f - 2 * K);
          if (canon >= 0) v = W_m[canon * H + i];
        }
        WmT[idx] = v;
      }
    }
  }
}

// ===========================================================================
// GEMM core: a WG tile of BN weight rows x BM activation rows, both operands
// staged through two LDS buffers, with global loads issued STAGES chunks
// ahead into a ring of register stages so their latency overlaps the MFMAs.
// Waves are laid out WAVES_M x WAVES_N x KSPLIT; the KSPLIT waves of one
// (wm, wn) position take interleaved MFMA K slices of every chunk and are
// summed through LDS at the end, so that only waves with kw == 0 hold the
// result.
//   acc[i][j] = W[n0 + (wn*NBW + i)*16 .. +16, :] . X[m0 + (wm*MBW + j)*16 .. +16, :]^T
// over K = Kpad columns; both sources address the tile's rows only.
// ===========================================================================
template <typename DT_, int NBW_, int MBW_, int WAVES_N_, int WAVES_M_, int KSPLIT_, int BK_,
          int STAGES_>
struct Gemm {
  using DT = DT_;
  static constexpr int NBW = NBW_, MBW = MBW_, WAVES_N = WAVES_N_, WAVES_M = WAVES_M_;
  static constexpr int KSPLIT = KSPLIT_, BK = BK_, STAGES = STAGES_;
  static constexpr int VEC = DType<DT>::VEC;
  static constexpr int NWAVES = WAVES_N * WAVES_M * KSPLIT;
  static constexpr int NT = 64 * NWAVES;
  static constexpr int BN = 16 * NBW * WAVES_N;
  static constexpr int BM = 16 * MBW * WAVES_M;
  // LDS rows padded by 32 bytes: 16-byte fragment reads of 16 rows at a
  // 160-byte stride run conflict-free on gfx950 (144 bytes: two-way conflicts)
  static constexpr int LDL = BK + 2 * VEC;
  static constexpr int KV = BK / VEC;   // 16-byte vectors per row chunk
  static constexpr int WV = BN * KV;
  static constexpr int XV = BM * KV;
  static constexpr int WIT = (WV + NT - 1) / NT;
  static constexpr int XIT = (XV + NT - 1) / NT;
  static constexpr int BUF = (BN + BM) * LDL;  // elements per LDS buffer
  static constexpr int NSLICE = BK / Mfma<DT>::KSLICE;
  static constexpr int RED_BYTES = (KSPLIT - 1) * WAVES_N * WAVES_M * NBW * MBW * 64 * 16;
  static constexpr int PIPE_BYTES = 2 * BUF * (int)sizeof(DT);
  static constexpr int LDS_BYTES = PIPE_BYTES > RED_BYTES ? PIPE_BYTES : RED_BYTES;
  static_assert(BK % Mfma<DT>::KSLICE == 0, "BK must be a multiple of the MFMA K slice");
  static_assert(NSLICE % KSPLIT == 0, "K slices must split evenly over the K waves");

  __device__ static int kw() { return (threadIdx.x >> 6) % KSPLIT; }
  __device__ static int wn() { return ((threadIdx.x >> 6) / KSPLIT) % WAVES_N; }
  __device__ static int wm() { return (threadIdx.x >> 6) / (KSPLIT * WAVES_N); }

  template <class S>
  __device__ __forceinline__ static void gload(uint4 (&wr)[WIT], uint4 (&xr)[XIT],
                                               const SrcX<DT>& w, const S& x, int Kpad, int k0) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int it = 0; it < WIT; ++it) {
      const int v = tid + it * NT;
      if (WV % NT == 0 || v < WV) wr[it] = w.load(w.row(v / KV), k0 + (v % KV) * VEC, Kpad);
    }
#pragma unroll
    for (int it = 0; it < XIT; ++it) {
      const int v = tid + it * NT;
      if (XV % NT == 0 || v < XV) xr[it] = x.load(x.row(v / KV), k0 + (v % KV) * VEC, Kpad);
    }
  }

  __device__ __forceinline__ static void sstore(const uint4 (&wr)[WIT], const uint4 (&xr)[XIT],
                                                DT* buf) {
    const int tid = threadIdx.x;
    DT* Xl = buf + BN * LDL;
#pragma unroll
    for (int it = 0; it < WIT; ++it) {
      const int v = tid + it * NT;
      if (WV % NT == 0 || v < WV)
        *reinterpret_cast<uint4*>(buf + (v / KV) * LDL + (v % KV) * VEC) = wr[it];
    }
#pragma unroll
    for (int it = 0; it < XIT; ++it) {
      const int v = tid + it * NT;
      if (XV % NT == 0 || v < XV)
        *reinterpret_cast<uint4*>(Xl + (v / KV) * LDL + (v % KV) * VEC) = xr[it];
    }
  }

  __device__ __forceinline__ static void compute(f32x4 (&acc)[NBW][MBW], const DT* buf) {
    const int lane = threadIdx.x & 63;
    const int g = lane >> 4, r16 = lane & 15;
    const int wni = wn(), wmi = wm();
    const DT* Xl = buf + BN * LDL;
    for (int sl = kw(); sl < NSLICE; sl += KSPLIT) {
      const int ks = sl * Mfma<DT>::KSLICE;
      uint4 a[NBW], b[MBW];
#pragma unroll
      for (int i = 0; i < NBW; ++i)
        a[i] = *reinterpret_cast<const uint4*>(buf + ((wni * NBW + i) * 16 + r16) * LDL + ks + g * VEC);
#pragma unroll
      for (int j = 0; j < MBW; ++j)
        b[j] = *reinterpret_cast<const uint4*>(Xl + ((wmi * MBW + j) * 16 + r16) * LDL + ks + g * VEC);
#pragma unroll
      for (int i = 0; i < NBW; ++i)
#pragma unroll
        for (int j = 0; j < MBW; ++j) Mfma<DT>::step(acc[i][j], a[i], b[j]);
    }
  }

  // w: weight rows n0 .. n0+BN-1; x: activation rows m0 .. m0+BM-1.
  template <class S>
  __device__ __forceinline__ static void run(f32x4 (&acc)[NBW][MBW], const SrcX<DT>& w, const S& x,
                                             int Kpad, DT* lds) {
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
      for (int j = 0; j < MBW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    uint4 wr[STAGES][WIT], xr[STAGES][XIT];
    const int nk = (Kpad + BK - 1) / BK;
#pragma unroll
    for (int s = 0; s < STAGES; ++s)
      if (s < nk) gload(wr[s], xr[s], w, x, Kpad, s * BK);
    sstore(wr[0], xr[0], lds);
    __syncthreads();
    for (int kc0 = 0; kc0 < nk; kc0 += STAGES) {
#pragma unroll
      for (int s = 0; s < STAGES; ++s) {
        const int kc = kc0 + s;
        if (kc < nk) {
          compute(acc, lds + (kc & 1) * BUF);
          if (kc + 1 < nk) sstore(wr[(s + 1) % STAGES], xr[(s + 1) % STAGES], lds + ((kc + 1) & 1) * BUF);
          if (kc + STAGES < nk) gload(wr[s], xr[s], w, x, Kpad, (kc + STAGES) * BK);
          __syncthreads();
        }
      }
    }
    if constexpr (KSPLIT > 1) {
      // sum the K partials into the kw == 0 waves (LDS is free after the loop)
      f32x4* red = reinterpret_cast<f32x4*>(lds);
      const int lane = threadIdx.x & 63;
      const int pos = wm() * WAVES_N + wn();
      const int k = kw();
      if (k > 0) {
#pragma unroll
        for (int i = 0; i < NBW; ++i)
#pragma unroll
          for (int j = 0; j < MBW; ++j)
            red[((((k - 1) * WAVES_N * WAVES_M + pos) * NBW + i) * MBW + j) * 64 + lane] = acc[i][j];
      }
      __syncthreads();
      if (k == 0) {
        for (int kk = 1; kk < KSPLIT; ++kk)
#pragma unroll
          for (int i = 0; i < NBW; ++i)
#pragma unroll
            for (int j = 0; j < MBW; ++j)
              acc[i][j] += red[((((kk - 1) * WAVES_N * WAVES_M + pos) * NBW + i) * MBW + j) * 64 + lane];
      }
      __syncthreads();
    }
  }
};

// ===========================================================================
// GEMM core for large row counts: operands go from global memory straight
// into LDS (buffer loads with the LDS-DMA modifier, no staging registers and
// no LDS store instructions, which on gfx950 run at about a third of the
// LDS read rate), through a ring of STAGES buffers so that the loads of
// chunk k + STAGES - 1 fly while chunk k is multiplied.  A chunk is 128 bytes
// of K per row (64 bf16 or 32 fp32 values, two MFMA K slices); rows are
// stored unpadded with their 16-byte pieces permuted, piece c of row r at
// slot c ^ ((r >> 1) & 7), which keeps the 16-row fragment reads free of
// bank conflicts.  One LDS-DMA instruction fills 8 rows (1 KB): lane l
// loads piece (l & 7) ^ ((row >> 1) & 7) of row 8q + (l >> 3).
// Same interface as Gemm (without a K split); Kpad must be a multiple of
// the chunk.
// ===========================================================================
struct NoWork {
  __device__ __forceinline__ void operator()() const {}
};

template <typename DT_, int NBW_, int MBW_, int WAVES_N_, int WAVES_M_, int STAGES_>
struct GemmD {
  using DT = DT_;
  static constexpr int NBW = NBW_, MBW = MBW_, WAVES_N = WAVES_N_, WAVES_M = WAVES_M_;
  static constexpr int STAGES = STAGES_, KSPLIT = 1;
  static constexpr int VEC = DType<DT>::VEC;
  static constexpr int BK = 128 / (int)sizeof(DT);  // K per chunk
  static constexpr int NWAVES = WAVES_N * WAVES_M;
  static constexpr int NT = 64 * NWAVES;
  static constexpr int BN = 16 * NBW * WAVES_N;
  static constexpr int BM = 16 * MBW * WAVES_M;
  static constexpr int ROWS = BN + BM;
  static constexpr int STAGE_BYTES = ROWS * 128;
  static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
  static constexpr int NQ = ROWS / 8;        // DMA instructions per chunk
  static constexpr int QW = NQ / NWAVES;     // ... per wave
  static_assert(NQ % NWAVES == 0 && BN % 8 == 0, "whole DMA instructions per wave");
  static_assert(STAGES >= 2 && (STAGES - 2) * QW < 64, "vmcnt range");
  static_assert(2 * Mfma<DT>::KSLICE == BK, "two MFMA K slices per chunk");

  __device__ static int kw() { return 0; }
  __device__ static int wn() { return (threadIdx.x >> 6) % WAVES_N; }
  __device__ static int wm() { return (threadIdx.x >> 6) / WAVES_N; }

  // this wave's chunks are in LDS once at most `young` later chunks are in flight
  __device__ __forceinline__ static void wait_chunks(int young) {
    if constexpr (STAGES >= 4) {
      if (young >= 2) { vm_wait<2 * QW>(); return; }
    }
    if constexpr (STAGES >= 3) {
      if (young >= 1) { vm_wait<QW>(); return; }
    }
    vm_wait<0>();
  }

  // GPERM: tile row 64 w + 16 i + 4 g + v of the weights is packed row
  // 64 w + 16 g + 4 v + i, so that with four 16-row blocks per wave, block i
  // of a wave holds gate i of 16 consecutive hidden units and lane (g, r16)
  // gets all four gates of units 4 g .. 4 g + 3 (the packed rows interleave
  // the gates per unit: row 4 u + q)
  // pre(): caller work that does not depend on the product, run once the
  // first chunks' loads are issued, so that it fills their latency
  template <class S, bool GPERM = false, class Pre = NoWork>
  __device__ __forceinline__ static void run(f32x4 (&acc)[NBW][MBW], const SrcX<DT>& w, const S& x,
                                             int Kpad, DT* lds, Pre&& pre = Pre{}) {
    static_assert(!S::kTwo, "the direct core reads one activation matrix");
    static_assert(!GPERM || NBW == 4, "the gate permutation needs four blocks per wave");
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 4, r16 = lane & 15;
    const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>(
        (__attribute__((address_space(3))) char*)reinterpret_cast<char*>(lds));
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
      for (int j = 0; j < MBW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // per-lane source offsets of this wave's DMA instructions (chunk 0); the
    // two buffer resources are selected per instruction rather than held in
    // one register quad each, which kept the scalar registers spilling
    const u32x4 rw = rsrc_words(w.base, w.bytes), rx = rsrc_words(x.base, x.bytes);
    bool isw[QW];
    uint32_t off[QW];
#pragma unroll
    for (int t = 0; t < QW; ++t) {
      const int q = wave * QW + t;  // uniform
      const int row = 8 * q + (lane >> 3);
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      isw[t] = q < BN / 8;
      const int wr = GPERM ? (row & ~63) | (((row >> 2) & 3) << 4) | ((row & 3) << 2) | ((row >> 4) & 3) : row;
      off[t] = isw[t] ? w.row(wr) + 16u * c : x.row(row - BN) + 16u * c;
    }
    const int nk = Kpad / BK;
    auto issue = [&](int kc) {
      const uint32_t base = lds0 + (uint32_t)(kc % STAGES) * STAGE_BYTES + (uint32_t)wave * QW * 1024u;
#pragma unroll
      for (int t = 0; t < QW; ++t) dma16(isw[t] ? rw : rx, off[t] + 128u * (uint32_t)kc, base + 1024u * t);
    };
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
      if (s < nk) issue(s);
    pre();

    const int wni = wn(), wmi = wm();
    const int sw = (r16 >> 1) & 7;
    const uint32_t col0 = (uint32_t)((g ^ sw) << 4), col1 = (uint32_t)(((4 + g) ^ sw) << 4);
    for (int kc = 0; kc < nk; ++kc) {
      wait_chunks(min(STAGES - 2, nk - 1 - kc));
      __builtin_amdgcn_s_barrier();  // no fence: it would wait for every load in flight
      asm volatile("" : : : "memory");
      if (kc + STAGES - 1 < nk) issue(kc + STAGES - 1);
      const char* buf = reinterpret_cast<const char*>(lds) + (kc % STAGES) * STAGE_BYTES;
#pragma unroll
      for (int sl = 0; sl < 2; ++sl) {
        const uint32_t col = sl ? col1 : col0;
        uint4 a[NBW], b[MBW];
#pragma unroll
        for (int i = 0; i < NBW; ++i)
          a[i] = *reinterpret_cast<const uint4*>(buf + ((wni * NBW + i) * 16 + r16) * 128 + col);
#pragma unroll
        for (int j = 0; j < MBW; ++j)
          b[j] = *reinterpret_cast<const uint4*>(buf + (BN + (wmi * MBW + j) * 16 + r16) * 128 + col);
#pragma unroll
        for (int i = 0; i < NBW; ++i)
#pragma unroll
          for (int j = 0; j < MBW; ++j) Mfma<DT>::step(acc[i][j], a[i], b[j]);
      }
    }
    __syncthreads();  // LDS free for the caller's epilogue
  }
};

template <class C> struct IsGemmD : std::false_type {};
template <typename DT, int NBW, int MBW, int WN, int WM, int ST>
struct IsGemmD<GemmD<DT, NBW, MBW, WN, WM, ST>> : std::true_type {};

// Static LDS a work-group may hold on gfx950 (160 KB per CU).
constexpr int kLdsStatic = 160 * 1024;

// Work-group -> tile mapping.  Work-groups are dispatched round-robin over
// the eight XCDs, each with its own L2.  The XCDs form a gn x (8 / gn) grid
// over (weight-row tiles, activation-row tiles): XCD x owns a contiguous
// range of nper weight tiles, so that its slice of the weights stays in its
// L2 across calls, and a range of mper activation tiles, which it walks
// with the weight tile fastest, so that an activation tile it has fetched
// is reused by all of its weight tiles while still in L2.  The host picks
// gn (tile_map below).  Returns false for padding work-groups.
struct TileMap {
  int nt, mt;      // weight-row tiles, activation-row tiles
  int gn;          // XCD groups along the weight tiles (1, 2, 4 or 8)
  int nper, mper;  // tiles of each kind per XCD
};

__device__ __forceinline__ bool tile_of(const TileMap& t, int& n, int& m) {
  const int x = blockIdx.x & 7, r = blockIdx.x >> 3;
  const int nl = r % t.nper, ml = r / t.nper;
  n = (x % t.gn) * t.nper + nl;
  m = (x / t.gn) * t.mper + ml;
  return n < t.nt && m < t.mt;
}

// ===========================================================================
// k_gates: g = W [q(z) | h]^T + WaT[a] + b, LSTM cell, commit.
// Rollout mode: a < 0 marks a frozen row, whose state is copied forward.
// NLL mode: every row is live; a outside [0, A) adds no column.
// ===========================================================================
struct GatesArgs {
  const void* Wg;
  const void* WaT;
  const float* bg;
  long ldk, ldx;
  int H, A, Z, M;
  const void* x_in;  // X_t [M, ldx] DT
  void* x_out;       // X_t+1 [M, ldx] DT: h_t+1 goes to columns Z .. Z+H-1
  float* c;          // [M, H] fp32, updated in place
  const int32_t* act;
  float* h_trace;  // [M, H] fp32 or null
  float* c_trace;
  int nll_mode;
  TileMap map;
};

// Element-wise side of the gate kernels for rows m0 .. m0+rows-1 of a tile.
// Every access goes through a range-checked buffer resource and elements
// that must not be touched get the offset kOffNone, so that the loads are
// straight-line code issued together, before any of their values is used.
// load() fetches what the cell needs besides the GEMM (bias plus the
// gathered one-hot column, cell state, and for a frozen row its h);
// commit() runs the LSTM cell on the four gate pre-activations i, f, g, o
// and stores h_t+1 into X_t+1 and c (a frozen rollout row keeps its state).
struct GateIn {
  float4 add;  // bias + one-hot column, per gate
  float c;     // cell state c_t
  float hprev; // h_t (frozen rows only)
  bool live;
};

template <typename DT>
struct GateIO {
  rsrc_t rc, rxi, rxo, rw, rb, rht, rct;
  int H, A;
  uint32_t ldxb;  // X row stride in bytes
  bool nll;

  __device__ GateIO(const GatesArgs& p, int m0, int rows) {
    H = p.H;
    A = p.A;
    nll = p.nll_mode != 0;
    const long mval = max(0, min(rows, p.M - m0));
    const uint32_t hb = (uint32_t)(mval * H * 4);
    ldxb = (uint32_t)(p.ldx * (long)sizeof(DT));
    const uint32_t xb = mval ? (uint32_t)(((mval - 1) * p.ldx + H) * (long)sizeof(DT)) : 0u;
    rc = make_rsrc(p.c + (long)m0 * H, hb);
    rxi = make_rsrc(reinterpret_cast<const DT*>(p.x_in) + (long)m0 * p.ldx + p.Z, xb);
    rxo = make_rsrc(reinterpret_cast<DT*>(p.x_out) + (long)m0 * p.ldx + p.Z, xb);
    rw = make_rsrc(p.WaT, (uint32_t)((long)A * 4 * H * (long)sizeof(DT)));
    rb = make_rsrc(p.bg, (uint32_t)(16 * H));
    rht = make_rsrc(p.h_trace ? p.h_trace + (long)m0 * H : nullptr, p.h_trace ? hb : 0u);
    rct = make_rsrc(p.c_trace ? p.c_trace + (long)m0 * H : nullptr, p.c_trace ? hb : 0u);
  }

  // tile row ml, hidden unit u, action a of the row; ok: inside the call
  __device__ __forceinline__ GateIn load(int ml, int u, int a, bool ok) const {
    GateIn in;
    in.live = nll || a >= 0;
    const uint32_t ec = ((uint32_t)ml * H + u) * 4u;
    const uint4 b = bload16(rb, ok ? (uint32_t)u * 16u : kOffNone);
    const bool gather = ok && a >= 0 && a < A;
    const uint32_t ew = ((uint32_t)a * 4u * H + 4u * u) * (uint32_t)sizeof(DT);
    float4 w;
    if constexpr (sizeof(DT) == 4) {
      const uint4 v = bload16(rw, gather ? ew : kOffNone);
      w = make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
    } else {
      const uint2 v = bload8(rw, gather ? ew : kOffNone);
      w = make_float4(bf16_bits_to_f32(v.x & 0xffffu), bf16_bits_to_f32(v.x >> 16),
                      bf16_bits_to_f32(v.y & 0xffffu), bf16_bits_to_f32(v.y >> 16));
    }
    in.add = make_float4(__uint_as_float(b.x) + w.x, __uint_as_float(b.y) + w.y,
                         __uint_as_float(b.z) + w.z, __uint_as_float(b.w) + w.w);
    in.c = __uint_as_float(bload4(rc, ok ? ec : kOffNone));
    const uint32_t ex = (uint32_t)ml * ldxb + (uint32_t)u * (uint32_t)sizeof(DT);
    const uint32_t ox = ok && !in.live ? ex : kOffNone;
    if constexpr (sizeof(DT) == 4) in.hprev = __uint_as_float(bload4(rxi, ox));
    else in.hprev = bf16_bits_to_f32(bload2(rxi, ox));
    return in;
  }

  __device__ __forceinline__ void commit(int ml, int u, bool ok, const GateIn& in, float pi, float pf,
                                         float pg, float po) const {
    const float cn = fsigmoid(pf + in.add.y) * in.c + fsigmoid(pi + in.add.x) * ftanh_cell<DT>(pg + in.add.z);
    const float hn = DType<DT>::round(fsigmoid(po + in.add.w) * ftanh_cell<DT>(cn));
    const float cv = in.live ? cn : in.c;
    const float hv = in.live ? hn : in.hprev;
    const uint32_t ec = ((uint32_t)ml * H + u) * 4u;
    const uint32_t ex = (uint32_t)ml * ldxb + (uint32_t)u * (uint32_t)sizeof(DT);
    bstore4(rc, ok && in.live ? ec : kOffNone, __float_as_uint(cv));
    if constexpr (sizeof(DT) == 4) bstore4(rxo, ok ? ex : kOffNone, __float_as_uint(hv));
    else bstore2(rxo, ok ? ex : kOffNone, f32_to_bf16_bits(hv));
    bstore4(rht, ok ? ec : kOffNone, __float_as_uint(hv));  // dropped without traces
    bstore4(rct, ok ? ec : kOffNone, __float_as_uint(cv));
  }
};

// Element-wise side of the pipelined gate kernels for four consecutive hidden
// units u0 .. u0+3 of one tile row, so that cell state, h, traces and the
// gathered one-hot columns move in 16-byte (8-byte for bf16 h) pieces.
// Same masking scheme as GateIO: range-checked buffer accesses, kOffNone for
// elements that must not be touched.
struct Gate4In {
  float4 add[4];  // bias + one-hot column of unit u0 + t, per gate
  float4 c;       // cell states of the four units
  float4 hprev;   // h_t of the four units (frozen rows only)
  bool live;
};

template <typename DT>
struct Gate4IO {
  rsrc_t rc, rxi, rxo, rw, rb, rht, rct;
  int H, A;
  uint32_t ldxb;
  bool nll, trace;

  __device__ Gate4IO(const GatesArgs& p, int m0, int rows) {
    H = p.H;
    A = p.A;
    nll = p.nll_mode != 0;
    trace = p.h_trace != nullptr;
    const long mval = max(0, min(rows, p.M - m0));
    const uint32_t hb = (uint32_t)(mval * H * 4);
    ldxb = (uint32_t)(p.ldx * (long)sizeof(DT));
    const uint32_t xb = mval ? (uint32_t)(((mval - 1) * p.ldx + H) * (long)sizeof(DT)) : 0u;
    rc = make_rsrc(p.c + (long)m0 * H, hb);
    rxi = make_rsrc(reinterpret_cast<const DT*>(p.x_in) + (long)m0 * p.ldx + p.Z, xb);
    rxo = make_rsrc(reinterpret_cast<DT*>(p.x_out) + (long)m0 * p.ldx + p.Z, xb);
    rw = make_rsrc(p.WaT, (uint32_t)((long)A * 4 * H * (long)sizeof(DT)));
    rb = make_rsrc(p.bg, (uint32_t)(16 * H));
    rht = make_rsrc(p.h_trace ? p.h_trace + (long)m0 * H : nullptr, p.h_trace ? hb : 0u);
    rct = make_rsrc(p.c_trace ? p.c_trace + (long)m0 * H : nullptr, p.c_trace ? hb : 0u);
  }

  // biases of units u0 .. u0+3 (gate order i, f, g, o)
  __device__ __forceinline__ void bias(int u0, bool ok, float4 (&b)[4]) const {
#pragma unroll
    for (int t = 0; t < 4; ++t) b[t] = as_float4(bload16(rb, ok ? (uint32_t)(u0 + t) * 16u : kOffNone));
  }

  // four 16-byte pieces of DT: units u0 .. u0+3 x 4 gates from WaT row a
  __device__ __forceinline__ void gather(uint32_t off, float4 (&w)[4]) const {
    if constexpr (sizeof(DT) == 4) {
#pragma unroll
      for (int t = 0; t < 4; ++t) w[t] = as_float4(bload16(rw, off == kOffNone ? kOffNone : off + 16u * t));
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4 v = bload16(rw, off == kOffNone ? kOffNone : off + 16u * h);
        w[2 * h] = make_float4(bf16_bits_to_f32(v.x & 0xffffu), bf16_bits_to_f32(v.x >> 16),
                               bf16_bits_to_f32(v.y & 0xffffu), bf16_bits_to_f32(v.y >> 16));
        w[2 * h + 1] = make_float4(bf16_bits_to_f32(v.z & 0xffffu), bf16_bits_to_f32(v.z >> 16),
                                   bf16_bits_to_f32(v.w & 0xffffu), bf16_bits_to_f32(v.w >> 16));
      }
    }
  }

  __device__ __forceinline__ Gate4In load(int ml, int u0, int a, bool ok, const float4 (&b)[4]) const {
    Gate4In in;
    in.live = nll || a >= 0;
    const bool gok = ok && a >= 0 && a < A;
    float4 w[4];
    gather(gok ? ((uint32_t)a * 4u * H + 4u * u0) * (uint32_t)sizeof(DT) : kOffNone, w);
#pragma unroll
    for (int t = 0; t < 4; ++t)
      in.add[t] = make_float4(b[t].x + w[t].x, b[t].y + w[t].y, b[t].z + w[t].z, b[t].w + w[t].w);
    in.c = as_float4(bload16(rc, ok ? ((uint32_t)ml * H + u0) * 4u : kOffNone));
    const uint32_t ox = ok && !in.live ? (uint32_t)ml * ldxb + (uint32_t)u0 * (uint32_t)sizeof(DT) : kOffNone;
    if constexpr (sizeof(DT) == 4) {
      in.hprev = as_float4(bload16(rxi, ox));
    } else {
      const uint2 v = bload8(rxi, ox);
      in.hprev = make_float4(bf16_bits_to_f32(v.x & 0xffffu), bf16_bits_to_f32(v.x >> 16),
                             bf16_bits_to_f32(v.y & 0xffffu), bf16_bits_to_f32(v.y >> 16));
    }
    return in;
  }

  // g[t]: GEMM part of the gates (i, f, g, o) of unit u0 + t
  __device__ __forceinline__ void commit(int ml, int u0, bool ok, const Gate4In& in, const float4 (&g)[4]) const {
    float cv[4], hv[4];
    const float cin[4] = {in.c.x, in.c.y, in.c.z, in.c.w};
    const float hin[4] = {in.hprev.x, in.hprev.y, in.hprev.z, in.hprev.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      float cn, hn;
      if constexpr (sizeof(DT) == 4) {
        cn = fsigmoid(g[t].y + in.add[t].y) * cin[t] + fsigmoid(g[t].x + in.add[t].x) * ftanh(g[t].z + in.add[t].z);
        hn = fsigmoid(g[t].w + in.add[t].w) * ftanh(cn);
      } else {
        lstm_cell_fused(g[t].x + in.add[t].x, g[t].y + in.add[t].y, g[t].z + in.add[t].z, g[t].w + in.add[t].w,
                        cin[t], cn, hn);
      }
      cv[t] = in.live ? cn : cin[t];
      hv[t] = in.live ? hn : hin[t];
    }
    const uint32_t ec = ((uint32_t)ml * H + u0) * 4u;
    const uint32_t ex = (uint32_t)ml * ldxb + (uint32_t)u0 * (uint32_t)sizeof(DT);
    const float4 c4 = make_float4(cv[0], cv[1], cv[2], cv[3]);
    bstore16(rc, ok && in.live ? ec : kOffNone, as_uint4(c4));
    float4 h4;
    if constexpr (sizeof(DT) == 4) {
      h4 = make_float4(hv[0], hv[1], hv[2], hv[3]);
      bstore16(rxo, ok ? ex : kOffNone, as_uint4(h4));
    } else {
      // h is stored rounded (a frozen row's h_t is already a bf16 value)
      const uint2 hb = make_uint2(pack2_bf16(hv[0], hv[1]), pack2_bf16(hv[2], hv[3]));
      bstore8(rxo, ok ? ex : kOffNone, hb);
      h4 = make_float4(bf16_bits_to_f32(hb.x & 0xffffu), bf16_bits_to_f32(hb.x >> 16),
                       bf16_bits_to_f32(hb.y & 0xffffu), bf16_bits_to_f32(hb.y >> 16));
    }
    if (trace) {
      bstore16(rht, ok ? ec : kOffNone, as_uint4(h4));
      bstore16(rct, ok ? ec : kOffNone, as_uint4(c4));
    }
  }
};

// Gate kernel on the pipelined cores.  The GEMM tile is staged through LDS
// as E[row][feature] (fp32) and the epilogue then runs with thread t on the
// four-unit group t % GPR of rows t / GPR, t / GPR + RSTEP, ...  A tile
// whose fp32 copy does not fit the LDS is staged in NPASS passes, one row of
// waves (PROWS tile rows) at a time.
template <class C>
__global__ void __launch_bounds__(C::NT) k_gates(const GatesArgs p) {
  using DT = typename C::DT;
  constexpr int NBW = C::NBW, MBW = C::MBW;
  constexpr int GPR = C::BN / 16;          // groups of four units per tile row
  constexpr int RSTEP = C::NT / GPR;       // rows per pass of the block
  constexpr int ELD = C::BN + 4;           // staged row stride (floats)
  constexpr int NPASS = C::BM * ELD * 4 <= kLdsStatic ? 1 : C::WAVES_M;
  constexpr int PROWS = C::BM / NPASS;     // tile rows staged per pass
  constexpr int IPT = (PROWS + RSTEP - 1) / RSTEP;
  constexpr int E_BYTES = PROWS * ELD * 4;
  constexpr int LDS = C::LDS_BYTES > E_BYTES ? C::LDS_BYTES : E_BYTES;
  static_assert(C::NT % GPR == 0, "whole groups per block");
  static_assert(NPASS == 1 || (E_BYTES <= kLdsStatic && C::KSPLIT == 1), "staged passes");
  __shared__ __attribute__((aligned(16))) char lds_raw[LDS];
  int nt, mt;
  if (!tile_of(p.map, nt, mt)) return;
  const int n0 = nt * C::BN, m0 = mt * C::BM;
  const int grp = threadIdx.x % GPR, r0 = threadIdx.x / GPR;
  const int u0 = n0 / 4 + 4 * grp;
  // actions of this thread's epilogue rows, fetched ahead of the GEMM
  int act[NPASS][IPT];
#pragma unroll
  for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
    for (int k = 0; k < IPT; ++k) {
      const int r = r0 + k * RSTEP, m = m0 + ps * PROWS + r;
      act[ps][k] = (r < PROWS && m < p.M) ? p.act[m] : -1;
    }
  const SrcX<DT> w(reinterpret_cast<const DT*>(p.Wg), p.ldk, p.ldk, n0, C::BN, 4 * p.H);
  const SrcX<DT> x(reinterpret_cast<const DT*>(p.x_in), p.ldx, p.ldx, m0, C::BM, p.M);
  f32x4 acc[NBW][MBW];
  C::run(acc, w, x, (int)p.ldk, reinterpret_cast<DT*>(lds_raw));

  float* E = reinterpret_cast<float*>(lds_raw);
  const Gate4IO<DT> io(p, m0, C::BM);
  const bool uok = u0 < p.H;  // H % 16 == 0: the whole group is inside
  float4 b[4];
  io.bias(u0, uok, b);
  // each pass's loads go out before its staging barrier, so that their
  // latency passes under the staging
  Gate4In in[IPT];
  auto load_pass = [&](int ps) {
    const int rp = ps * PROWS;  // first tile row of the pass
#pragma unroll
    for (int k = 0; k < IPT; ++k) {
      const int r = r0 + k * RSTEP;
      in[k] = io.load(rp + r, u0, act[ps][k], uok && r < PROWS && m0 + rp + r < p.M, b);
    }
  };
  load_pass(0);
#pragma unroll
  for (int ps = 0; ps < NPASS; ++ps) {
    if (ps > 0) {
      load_pass(ps);
      __syncthreads();  // the previous pass has read E
    }
    if (C::kw() == 0 && (NPASS == 1 || C::wm() == ps)) {
      const int lane = threadIdx.x & 63, r16 = lane & 15, g = lane >> 4;
      const int wn = C::wn(), wmi = NPASS == 1 ? C::wm() : 0;
#pragma unroll
      for (int j = 0; j < MBW; ++j)
#pragma unroll
        for (int i = 0; i < NBW; ++i)
          *reinterpret_cast<f32x4*>(E + ((wmi * MBW + j) * 16 + r16) * ELD + (wn * NBW + i) * 16 + 4 * g) =
              acc[i][j];
    }
    __syncthreads();

    const int rp = ps * PROWS;  // first tile row of the pass
#pragma unroll
    for (int k = 0; k < IPT; ++k) {
      const int r = r0 + k * RSTEP;
      if (r >= PROWS) continue;
      float4 gsum[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) gsum[t] = *reinterpret_cast<const float4*>(E + r * ELD + 16 * grp + 4 * t);
      io.commit(rp + r, u0, uok && m0 + rp + r < p.M, in[k], gsum);
    }
  }
}

// Gate kernel with the epilogue straight from the MFMA accumulators (four
// 16-row blocks per wave, no split K): the weight tile is loaded with the
// gate permutation of GemmD::run, so lane (g, r16) holds, in acc[q][j][v],
// gate q of unit n0/4 + 16 wn + 4 g + v for row (wm MBW + j) 16 + r16 of the
// tile.  Each lane then runs the LSTM cell of four consecutive units of its
// MBW rows, with the next row's loads in flight under the current row's
// cell; no LDS staging, no barrier after the GEMM.
template <class C>
__global__ void __launch_bounds__(C::NT) k_gates_direct(const GatesArgs p) {
  using DT = typename C::DT;
  constexpr int MBW = C::MBW;
  static_assert(C::NBW == 4 && C::KSPLIT == 1, "four gate blocks per wave");
  __shared__ __attribute__((aligned(16))) char lds_raw[C::LDS_BYTES];
  int nt, mt;
  if (!tile_of(p.map, nt, mt)) return;
  const int n0 = nt * C::BN, m0 = mt * C::BM;
  const int lane = threadIdx.x & 63, g = lane >> 4, r16 = lane & 15;
  const int wn = C::wn(), wmi = C::wm();
  const int u0 = n0 / 4 + 16 * wn + 4 * g;  // this lane's four units
  // the lane's rows and their actions, fetched ahead of the GEMM
  int act[MBW];
#pragma unroll
  for (int j = 0; j < MBW; ++j) {
    const int m = m0 + (wmi * MBW + j) * 16 + r16;
    act[j] = m < p.M ? p.act[m] : -1;
  }
  const SrcX<DT> w(reinterpret_cast<const DT*>(p.Wg), p.ldk, p.ldk, n0, C::BN, 4 * p.H);
  const SrcX<DT> x(reinterpret_cast<const DT*>(p.x_in), p.ldx, p.ldx, m0, C::BM, p.M);
  f32x4 acc[4][MBW];
  C::template run<SrcX<DT>, true>(acc, w, x, (int)p.ldk, reinterpret_cast<DT*>(lds_raw));

  const Gate4IO<DT> io(p, m0, C::BM);
  const bool uok = u0 < p.H;  // H % 16 == 0: the four units are inside together
  float4 b[4];
  io.bias(u0, uok, b);
  auto row_of = [&](int j) { return (wmi * MBW + j) * 16 + r16; };
  auto ok_of = [&](int j) { return uok && m0 + row_of(j) < p.M; };
  Gate4In cur = io.load(row_of(0), u0, act[0], ok_of(0), b);
#pragma unroll
  for (int j = 0; j < MBW; ++j) {
    Gate4In nxt;
    if (j + 1 < MBW) nxt = io.load(row_of(j + 1), u0, act[j + 1], ok_of(j + 1), b);
    float4 gs[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) gs[t] = make_float4(acc[0][j][t], acc[1][j][t], acc[2][j][t], acc[3][j][t]);
    io.commit(row_of(j), u0, ok_of(j), cur, gs);
    if (j + 1 < MBW) cur = nxt;
  }
}

// ===========================================================================
// k_mdn: mixture head on h_{t+1}.  Each wave owns one group of four latent
// dims (Q output blocks), so each lane holds all features of one dim.
// Rollout epilogue: component pick + Box-Muller + z commit.
// NLL epilogue: per-dim log-likelihood, summed over the tile's dims; the
// extra last tile column computes the reward / done logits.
// ===========================================================================
struct MdnArgs {
  const void* Wm;
  const float* bm;
  long ldh, ldx;
  int H, Z, K, Nm, M;
  // [M, ldx] DT activation rows: the head reads h at columns Z ..; the
  // rollout writes q(z_t+1) to columns 0 .. Z-1
  void* x;
  // rollout
  const int32_t* act;
  const float* z_prev;  // [M, Z]
  float* z_next;        // [M, Z]
  uint32_t k0, k1, step, traj0;
  float tau;
  float sig;  // scale of the normal deviate: sqrt(tau) with the sigma temperature, else 1
  // nll
  const float* z_tgt;  // [M, Z]
  float* part;         // [M, ntd]
  float* head;         // [M, 2]
  int ntd;
  int nll_mode;
  TileMap map;
};

// z_{t+1,j} of row m (mixture_noise / mixture_pick with the call's step,
// temperature and trajectory index).
__device__ __forceinline__ MdnNoise mdn_noise(const MdnArgs& p, const Rng& rng, int m, int j, int K) {
  return mixture_noise(rng, K, p.step, p.traj0 + (uint32_t)m, j);
}

template <int Q>
__device__ __forceinline__ float mdn_pick(const MdnArgs& p, const MdnNoise& n,
                                          const float (&feat)[4 * Q], int K) {
  return mixture_pick<Q>(K, p.tau, n, feat, p.sig);
}

template <int Q>
__device__ __forceinline__ float mdn_draw(const MdnArgs& p, const Rng& rng, int m, int j,
                                          const float (&feat)[4 * Q], int K) {
  return mdn_pick<Q>(p, mdn_noise(p, rng, m, j, K), feat, K);
}

// log sum_k pi_k N(x; mu_k, sigma_k) of one latent dim (pi at tau = 1).
template <int Q>
__device__ __forceinline__ float mdn_loglik(float x, const float (&feat)[4 * Q], int K) {
  float mx = -INFINITY;
#pragma unroll
  for (int f = 0; f < 4 * Q; ++f)
    if (f < K) mx = fmaxf(mx, feat[f]);
  float se = 0.f;
#pragma unroll
  for (int f = 0; f < 4 * Q; ++f)
    if (f < K) se += expf(feat[f] - mx);
  const float lse_pi = mx + logf(se);
  float terms[4 * Q];
  float tmax = -INFINITY;
#pragma unroll
  for (int f = 0; f < 4 * Q; ++f) {
    terms[f] = -INFINITY;
    if (f < K) {
      float mu = 0.f, ls = 0.f;
#pragma unroll
      for (int f2 = 0; f2 < 4 * Q; ++f2) {
        if (f2 == K + f) mu = feat[f2];
        if (f2 == 2 * K + f) ls = feat[f2];
      }
      const float d = (x - mu) * expf(-ls);
      terms[f] = (feat[f] - lse_pi) - 0.5f * d * d - ls - kHalfLn2Pi;
      tmax = fmaxf(tmax, terms[f]);
    }
  }
  float st = 0.f;
#pragma unroll
  for (int f = 0; f < 4 * Q; ++f)
    if (f < K) st += expf(terms[f] - tmax);
  return tmax + logf(st);
}

// z_{t+1,j} of row m goes to the fp32 output and, rounded, to X_{t+1}.
template <typename DT>
__device__ __forceinline__ void mdn_commit(const MdnArgs& p, int m, int j, float z) {
  p.z_next[(long)m * p.Z + j] = z;
  DType<DT>::store(reinterpret_cast<DT*>(p.x), (long)m * p.ldx + j, z);
}

// KC: the number of mixture components (the call's K), a compile-time
// constant so that the feature selections of the epilogue fold away
template <class C, int KC>
__global__ void __launch_bounds__(C::NT) k_mdn(const MdnArgs p) {
  using DT = typename C::DT;
  constexpr int K = KC;
  constexpr int Q = C::NBW, MBW = C::MBW, WAVES_N = C::WAVES_N, WAVES_M = C::WAVES_M;
  static_assert(WAVES_N == 2, "the NLL epilogue sums two dim groups per work-group");
  __shared__ __attribute__((aligned(16))) char lds_raw[C::LDS_BYTES];
  // NLL partial sums of the second dim group; reuses the GEMM's LDS, which
  // is free once run() has returned
  float(*red)[MBW * 16] = reinterpret_cast<float(*)[MBW * 16]>(lds_raw);
  static_assert(WAVES_M * MBW * 16 * 4 <= C::LDS_BYTES, "partial sums fit the GEMM's LDS");
  int ntile, mt;
  if (!tile_of(p.map, ntile, mt)) return;
  const int n0 = ntile * C::BN, m0 = mt * C::BM;
  const int lane = threadIdx.x & 63;
  const int wn = C::wn(), wmi = C::wm();
  const int g = lane >> 4;
  const int Z = p.Z;
  const int J = ntile * WAVES_N + wn;  // dim group of this wave
  const int j = 4 * J + g;             // latent dim of this lane
  const bool head_tile = p.nll_mode && ntile == p.ntd;
  // rollout: the actions of this lane's rows and their previous latents
  // (kept by frozen rows), fetched ahead of the GEMM
  int actp[MBW];
  float zpv[MBW];
  if (!p.nll_mode) {
    const long mval = max(0, min(C::BM, p.M - m0));
    const rsrc_t ra = make_rsrc(p.act + m0, (uint32_t)(mval * 4));
    const rsrc_t rz = make_rsrc(p.z_prev + (long)m0 * Z, (uint32_t)(mval * Z * 4));
#pragma unroll
    for (int jj = 0; jj < MBW; ++jj) {
      const int ml = (wmi * MBW + jj) * 16 + (lane & 15);
      const bool ok = m0 + ml < p.M && j < Z;
      actp[jj] = (int)bload4(ra, ok ? (uint32_t)ml * 4u : kOffNone);
      zpv[jj] = __uint_as_float(bload4(rz, ok ? (uint32_t)(ml * Z + j) * 4u : kOffNone));
    }
  }
  const SrcX<DT> w(reinterpret_cast<const DT*>(p.Wm), p.ldh, p.ldh, n0, C::BN, p.Nm);
  const SrcX<DT> x(reinterpret_cast<const DT*>(p.x) + p.Z, p.ldx, p.ldx - p.Z, m0, C::BM, p.M);
  const Rng rng{p.k0, p.k1};
  // The four lanes of a row (lane groups g, dims 4J + g) need the same
  // stream-2 block.  With four row blocks per lane, lane group g draws the
  // block and both Box-Muller pairs for row block g only, and every lane
  // reads its deviates from the drawing lanes (shuffles, all lanes active),
  // instead of each lane drawing all four blocks.  On the direct core these
  // draws run while the GEMM's first chunks load: they do not depend on the
  // product.  (Drawing the component noise there too, for every row, frozen
  // or not, made the xlarge mixture kernel slower: 108.7 against 107.3 us.)
  constexpr bool kPre = IsGemmD<C>::value && MBW == 4;
  float eps[MBW];
  auto draw_eps = [&]() {
    if constexpr (MBW == 4) {
      const float4 e = gauss_group(rng, p.step, p.traj0 + (uint32_t)(m0 + (wmi * MBW + g) * 16 + (lane & 15)), J);
#pragma unroll
      for (int jj = 0; jj < MBW; ++jj) {
        const int src = jj * 16 + (lane & 15);
        const float v0 = __shfl(e.x, src), v1 = __shfl(e.y, src), v2 = __shfl(e.z, src), v3 = __shfl(e.w, src);
        eps[jj] = g == 0 ? v0 : (g == 1 ? v1 : (g == 2 ? v2 : v3));
      }
    }
  };
  auto pre = [&]() {
    if (!p.nll_mode) draw_eps();
  };
  f32x4 acc[Q][MBW];
  if constexpr (kPre)
    C::run(acc, w, x, (int)p.ldh, reinterpret_cast<DT*>(lds_raw), pre);
  else
    C::run(acc, w, x, (int)p.ldh, reinterpret_cast<DT*>(lds_raw));
  const bool owner = C::kw() == 0;  // holds the summed tile

  if (head_tile) {
    // Rows 0 and 1 of the block are the reward and done logits.
    if (owner && wn == 0 && g == 0) {
#pragma unroll
      for (int jj = 0; jj < MBW; ++jj) {
        const int m = m0 + (wmi * MBW + jj) * 16 + (lane & 15);
        if (m < p.M) {
          p.head[2 * (long)m] = acc[0][jj][0] + p.bm[n0];
          p.head[2 * (long)m + 1] = acc[0][jj][1] + p.bm[n0 + 1];
        }
      }
    }
    return;
  }

  // features f = 4q + v of dim j: acc[q][.][v] + bias
  float bias[4 * Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const float4 b4 = *reinterpret_cast<const float4*>(p.bm + J * 16 * Q + 16 * q + 4 * g);
    bias[4 * q] = b4.x; bias[4 * q + 1] = b4.y; bias[4 * q + 2] = b4.z; bias[4 * q + 3] = b4.w;
  }

  if (!p.nll_mode) {
    if (!owner) return;  // no barrier below
    if constexpr (!kPre) draw_eps();
#pragma unroll
    for (int jj = 0; jj < MBW; ++jj) {
      const int m = m0 + (wmi * MBW + jj) * 16 + (lane & 15);
      if (m >= p.M || j >= Z) continue;
      if (actp[jj] < 0) {
        mdn_commit<DT>(p, m, j, zpv[jj]);
        continue;
      }
      float feat[4 * Q];
#pragma unroll
      for (int q = 0; q < Q; ++q)
#pragma unroll
        for (int v = 0; v < 4; ++v) feat[4 * q + v] = acc[q][jj][v] + bias[4 * q + v];
      if constexpr (MBW == 4) {
        MdnNoise nz;
        component_noise(nz, rng, K, p.step, p.traj0 + (uint32_t)m, j);
        nz.eps = eps[jj];
        mdn_commit<DT>(p, m, j, mdn_pick<Q>(p, nz, feat, K));
      } else {
        mdn_commit<DT>(p, m, j, mdn_draw<Q>(p, rng, m, j, feat, K));
      }
    }
  } else {
#pragma unroll
    for (int jj = 0; jj < MBW; ++jj) {
      const int m = m0 + (wmi * MBW + jj) * 16 + (lane & 15);
      float ll = 0.f;
      if (owner && m < p.M && j < Z) {
        float feat[4 * Q];
#pragma unroll
        for (int q = 0; q < Q; ++q)
#pragma unroll
          for (int v = 0; v < 4; ++v) feat[4 * q + v] = acc[q][jj][v] + bias[4 * q + v];
        ll = mdn_loglik<Q>(p.z_tgt[(long)m * Z + j], feat, K);
      }
      // sum over the four dims of the group (lane groups), then the two waves
      ll += __shfl_xor(ll, 16);
      ll += __shfl_xor(ll, 32);
      if (owner && wn == 1 && g == 0) red[wmi][jj * 16 + (lane & 15)] = ll;
      __syncthreads();
      if (owner && wn == 0 && g == 0 && m < p.M)
        p.part[(long)m * p.ntd + ntile] = ll + red[wmi][jj * 16 + (lane & 15)];
      __syncthreads();
    }
  }
}

// ===========================================================================
// k_ctrl: controller logits for BM = 16*MBW rows (all Nc outputs in one
// block; four waves take interleaved 16-output slices), weights read
// straight from global memory, activations staged through LDS in K chunks.
//   mode 0: controller step (probs + action)
//   mode 1: rollout step t: resolve transition t-1, choose a_t
//   mode 2: rollout tail: resolve transition T-1 only
// ===========================================================================
struct CtrlArgs {
  const void* Wc;
  const float* bc;
  long ldk;
  int Z, H, A, Nc, M;
  const void* x;   // rollout: X_t [M, ldx] DT
  long ldx;
  const float* z;  // controller step: z [M, Z] and h [M, H], fp32
  const float* h;
  const uint8_t* mask;
  uint32_t k0, k1, step, traj0;
  int mode;
  // mode 0
  float* probs;
  int32_t* action;
  // mode 1/2
  int32_t* act_t;       // [M]
  const int32_t* act_prev;  // [M] or null (t == 0)
  float* rew_prev;
  uint8_t* done_prev;
  float* rew_t;
  uint8_t* done_t;
  int32_t* done_state;
  int use_done;
  // per-trajectory horizons (null: T for all): a step t >= lengths[m] is padding
  const int32_t* lengths;
  int t;
  // two-level controller (N > 0): mask holds the xfer masks [M, N+1]
  // followed by the location masks [M, N, Lc]; the logits are the N+1 xfer
  // rows then the Lc location rows
  int N, Lc;
  // logits stored instead of picked (k_ctrl_wide): columns [0, ncol) of each
  // row, bias not added, at logits_out + m ldl; k_ctrl_rows then picks
  float* logits_out;
  long ldl;
  int ncol;
  float* lg_ws;  // rollout workspace [M, Nc] for those logits (wide two-level controllers)
};

// Rollout bookkeeping of row m at step t (modes 1 and 2 of the controller
// kernels).  First the previous transition t-1 is resolved if the row was
// live then: its reward is the reward head on h_t and it is done when
// sigmoid(done head) exceeds the stream-3 uniform of step t-1.  Then (mode 1)
// the row takes action `a` (the masked Gumbel-max, -1 if no action is valid)
// or, if done, the frozen outputs; a row without a valid action ends here.
// A step past the row's horizon is padding: no action, reward 0, done 0 (its
// state is kept like a frozen row's; the latent is zeroed afterwards).
__device__ __forceinline__ void ctrl_row_commit(const CtrlArgs& p, const Rng& rng, int m, int a,
                                                float rr, float rd) {
  int ds = p.done_state[m];
  if (p.act_prev && p.act_prev[m] >= 0) {
    p.rew_prev[m] = rr;
    int d = 0;
    if (p.use_done) {
      const uint4 w = rng.block(0, p.step - 1u, p.traj0 + (uint32_t)m, STREAM_DONE);
      d = sigmoidf(rd) > word_to_uniform(w.x);
    }
    p.done_prev[m] = (uint8_t)d;
    if (d) ds = 1;
  }
  if (p.mode == 1) {
    const bool pad = p.lengths && p.t >= p.lengths[m];
    if (ds || pad) a = -1;
    else if (a < 0) ds = 1;
    p.act_t[m] = a;
    if (a < 0) {
      p.rew_t[m] = 0.f;
      p.done_t[m] = pad ? 0 : 1;
    }
  }
  p.done_state[m] = ds;
}

// Two-level pick of row m (section 3.1.3) by its TPR threads (thread q of
// the row), from its logits lg (bias not yet added): an xfer among the valid
// ones (stream 0, index x; x = N is the NO-OP), then a location valid for
// that xfer (stream 4, index l).  two_level_xfer returns x (-1 when none is
// valid), two_level_loc the location of xfer x < N (-1 when none is valid),
// two_level_pick the flat action x Lc + l, -2 for the NO-OP, -1 when nothing
// is valid; the same value in every thread of the row.  Ties go to the
// lowest index.  LMAX bounds Lc.
template <int TPR>
__device__ __forceinline__ void row_argmax(float& best, int& bidx) {
#pragma unroll
  for (int off = 1; off < TPR; off <<= 1) {
    const float ob = __shfl_xor(best, off);
    const int oi = __shfl_xor(bidx, off);
    if (oi >= 0 && (bidx < 0 || ob > best || (ob == best && oi < bidx))) { best = ob; bidx = oi; }
  }
}

template <int TPR>
__device__ __forceinline__ int two_level_xfer(const CtrlArgs& p, const Rng& rng, const float* lg, int m,
                                              bool on, int q, uint32_t traj) {
  const int NX = p.N + 1;
  float best = -INFINITY;
  int x = -1;
  if (on) {
    for (int i = q; i < NX; i += TPR) {
      if (!p.mask[(long)m * NX + i]) continue;
      const uint4 w = rng.block((uint32_t)i >> 2, p.step, traj, STREAM_CONTROLLER);
      const float sc = lg[i] + p.bc[i] + gumbel(word_to_uniform(word_of(w, i & 3)));
      if (sc > best) { best = sc; x = i; }
    }
  }
  row_argmax<TPR>(best, x);
  return x;
}

template <int TPR, int LMAX>
__device__ __forceinline__ int two_level_loc(const CtrlArgs& p, const Rng& rng, const float* lg, int m,
                                             bool on, int q, uint32_t traj, int x) {
  const int N = p.N, NX = N + 1, Lc = p.Lc;
  const uint8_t* lm = p.mask + (long)p.M * NX + ((long)m * N + x) * Lc;
  // thread q takes the contiguous locations [l0, l1) (a multiple of four:
  // one Philox block each); their mask bytes are all loaded before the
  // first is used, instead of one dependent load per location
  constexpr int MAXW = (((LMAX + TPR - 1) / TPR + 3) & ~3) / 4;
  const int cpt = ((Lc + TPR - 1) / TPR + 3) & ~3;
  const int l0 = q * cpt, l1 = min(l0 + cpt, Lc);
  uint32_t mw[MAXW];
#pragma unroll
  for (int k = 0; k < MAXW; ++k) {
    uint32_t wv = 0;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = l0 + 4 * k + v;
      if (on && i < l1 && lm[i]) wv |= 1u << (8 * v);
    }
    mw[k] = wv;
  }
  float best = -INFINITY;
  int l = -1;
#pragma unroll
  for (int k = 0; k < MAXW; ++k) {
    if (mw[k] == 0) continue;
    const int b = l0 + 4 * k;
    const uint4 w = rng.block((uint32_t)b >> 2, p.step, traj, STREAM_LOCATION);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if ((mw[k] >> (8 * v)) & 1u) {
        const float sc = lg[NX + b + v] + p.bc[NX + b + v] + gumbel(word_to_uniform(word_of(w, v)));
        if (sc > best) { best = sc; l = b + v; }
      }
    }
  }
  row_argmax<TPR>(best, l);
  return l;
}

template <int TPR, int LMAX = 316>
__device__ __forceinline__ int two_level_pick(const CtrlArgs& p, const Rng& rng, const float* lg,
                                              int m, bool on, int q, uint32_t traj) {
  const int x = two_level_xfer<TPR>(p, rng, lg, m, on, q, traj);
  if (x < 0) return -1;
  if (x == p.N) return -2;
  const int l = two_level_loc<TPR, LMAX>(p, rng, lg, m, on, q, traj, x);
  return l < 0 ? -1 : x * p.Lc + l;
}

// The two-level controller from stored logits (k_ctrl_wide with logits_out),
// one wave per row, for controllers too wide for the staged tiles and for
// the controller step.  Rollout modes: the pick and the row's commit (the
// reward and done logits are columns Ac, Ac + 1).  Mode 0: the action and,
// over the row's logits in place, the probabilities: the softmax of the
// valid xfers' logits [N+1], then the softmax of the valid locations of the
// picked xfer [Lc] (0 after a NO-OP or when nothing is valid).
constexpr int kRowsMax = 1024;  // N + 1 and Lc at most this
__global__ void __launch_bounds__(256) k_ctrl_rows(const CtrlArgs p) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (m >= p.M) return;  // the whole wave
  float* lg = p.logits_out + (long)m * p.ldl;
  const Rng rng{p.k0, p.k1};
  const uint32_t traj = p.traj0 + (uint32_t)m;
  const int N = p.N, NX = N + 1, Lc = p.Lc;
  if (p.mode != 0) {
    int a = -1;
    if (p.mode == 1) {
      const int x = two_level_xfer<64>(p, rng, lg, m, true, lane, traj);
      if (x == N) a = -2;
      else if (x >= 0) {
        const int l = two_level_loc<64, kRowsMax>(p, rng, lg, m, true, lane, traj, x);
        a = l < 0 ? -1 : x * Lc + l;
      }
    }
    const int Ar = NX + Lc;
    if (lane == 0) ctrl_row_commit(p, rng, m, a, lg[Ar] + p.bc[Ar], lg[Ar + 1] + p.bc[Ar + 1]);
    return;
  }
  const int x = two_level_xfer<64>(p, rng, lg, m, true, lane, traj);
  const bool locs = x >= 0 && x < N;
  const int l = locs ? two_level_loc<64, kRowsMax>(p, rng, lg, m, true, lane, traj, x) : -1;
  const int a = x < 0 ? -1 : x == N ? -2 : l < 0 ? -1 : x * Lc + l;
  // every logit this lane needs, read before any probability is written
  constexpr int PER = kRowsMax / 64;
  const uint8_t* lm = p.mask + (long)p.M * NX + ((long)m * N + (locs ? x : 0)) * Lc;
  float vx[PER], vl[PER];
  float mxx = -INFINITY, mxl = -INFINITY;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int i = lane + 64 * k;
    const bool okx = i < NX && p.mask[(long)m * NX + i];
    vx[k] = okx ? lg[i] + p.bc[i] : -INFINITY;
    mxx = fmaxf(mxx, vx[k]);
    const bool okl = locs && i < Lc && lm[i];
    vl[k] = okl ? lg[NX + i] + p.bc[NX + i] : -INFINITY;
    mxl = fmaxf(mxl, vl[k]);
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    mxx = fmaxf(mxx, __shfl_xor(mxx, off));
    mxl = fmaxf(mxl, __shfl_xor(mxl, off));
  }
  float sx = 0.f, sl = 0.f;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    vx[k] = vx[k] == -INFINITY ? 0.f : expf(vx[k] - mxx);
    vl[k] = vl[k] == -INFINITY ? 0.f : expf(vl[k] - mxl);
    sx += vx[k];
    sl += vl[k];
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    sx += __shfl_xor(sx, off);
    sl += __shfl_xor(sl, off);
  }
  const float ix = sx > 0.f ? 1.0f / sx : 0.f, il = sl > 0.f ? 1.0f / sl : 0.f;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int i = lane + 64 * k;
    if (i < NX) lg[i] = vx[k] * ix;
    if (i < Lc) lg[NX + i] = vl[k] * il;
  }
  if (lane == 0) p.action[m] = a;
}

// Activation source of the controller kernels for rows m0 .. m0+rows-1.
template <class S>
__device__ __forceinline__ S ctrl_src(const CtrlArgs& p, int m0, int rows) {
  using DT = typename S::DT;
  if constexpr (S::kTwo) return S(p.z, p.h, p.Z, p.H, m0, rows, p.M);
  else return S(reinterpret_cast<const DT*>(p.x), p.ldx, p.ldx, m0, rows, p.M);
}

template <class S, int NBW, int MBW, int BKC>
__global__ void __launch_bounds__(256) k_ctrl_wide(const CtrlArgs p) {
  using DT = typename S::DT;
  constexpr int VEC = DType<DT>::VEC;
  constexpr int BM = 16 * MBW;
  constexpr int LDL = BKC + 2 * VEC;
  __shared__ __attribute__((aligned(16))) DT xl[BM * LDL];
  __shared__ float s_best[4][BM];
  __shared__ int s_idx[4][BM];
  __shared__ float s_max[4][BM];
  __shared__ float s_rho[BM][2];
  __shared__ float s_fin[BM][2];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, r16 = lane & 15;
  const int m0 = blockIdx.x * BM;
  const int nbtot = p.Nc / 16;
  const DT* W = reinterpret_cast<const DT*>(p.Wc);
  const S src = ctrl_src<S>(p, m0, BM);

  f32x4 acc[NBW][MBW];
#pragma unroll
  for (int i = 0; i < NBW; ++i)
#pragma unroll
    for (int j = 0; j < MBW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kc = 0; kc < (int)p.ldk; kc += BKC) {
    __syncthreads();
    for (int v = tid; v < BM * (BKC / VEC); v += 256) {
      const int r = v / (BKC / VEC), kv = v % (BKC / VEC);
      *reinterpret_cast<uint4*>(xl + r * LDL + kv * VEC) = src.load(src.row(r), kc + kv * VEC, (int)p.ldk);
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < BKC; ks += Mfma<DT>::KSLICE) {
      if (kc + ks >= (int)p.ldk) break;  // last chunk may overhang the padded K
      // the slice's weight fragments are loaded in groups of GW, one group
      // ahead of its MFMAs, from rows clamped into the matrix (blocks past
      // nbtot are loaded but not used). Unguarded loads let each MFMA wait
      // for its own fragment only; under the guard it waited for all of them.
      constexpr int GW = 8, NG = (NBW + GW - 1) / GW;
      uint4 a[2][GW];
      auto load_group = [&](int gi, uint4(&dst)[GW]) {
#pragma unroll
        for (int q = 0; q < GW; ++q) {
          const int i = gi * GW + q;
          if (i < NBW) {
            const int nb = min(wave + 4 * i, nbtot - 1);
            dst[q] = *reinterpret_cast<const uint4*>(W + (long)(nb * 16 + r16) * p.ldk + kc + ks + g * VEC);
          }
        }
      };
      load_group(0, a[0]);
      uint4 b[MBW];
#pragma unroll
      for (int j = 0; j < MBW; ++j)
        b[j] = *reinterpret_cast<const uint4*>(xl + (j * 16 + r16) * LDL + ks + g * VEC);
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        if (gi + 1 < NG) load_group(gi + 1, a[(gi + 1) & 1]);
#pragma unroll
        for (int q = 0; q < GW; ++q) {
          const int i = gi * GW + q;
          if (i < NBW && wave + 4 * i < nbtot) {
#pragma unroll
            for (int j = 0; j < MBW; ++j) Mfma<DT>::step(acc[i][j], a[gi & 1][q], b[j]);
          }
        }
      }
    }
  }

  // ---- epilogue ----
  if (p.logits_out) {  // logits only (bias not added); k_ctrl_rows picks
#pragma unroll
    for (int j = 0; j < MBW; ++j) {
      const int m = m0 + j * 16 + r16;
      if (m >= p.M) continue;
#pragma unroll
      for (int i = 0; i < NBW; ++i) {
        const int nb = wave + 4 * i;
        const int n = nb * 16 + 4 * g;
        if (nb >= nbtot) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (n + v < p.ncol) p.logits_out[(long)m * p.ldl + n + v] = acc[i][j][v];
      }
    }
    return;
  }
  const Rng rng{p.k0, p.k1};
  const int A = p.A;
  const bool want_action = p.mode != 2;
  // the mask bytes of this lane's actions (n .. n+3 of each block, each
  // row), all loaded before the first is used
  uint32_t mk[NBW][MBW];
#pragma unroll
  for (int j = 0; j < MBW; ++j) {
    const int m = m0 + j * 16 + r16;
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
      const int n = (wave + 4 * i) * 16 + 4 * g;
      uint32_t wv = 0;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (m < p.M && wave + 4 * i < nbtot && n + v < A && p.mask[(long)m * A + n + v]) wv |= 1u << (8 * v);
      mk[i][j] = wv;
    }
  }
#pragma unroll
  for (int j = 0; j < MBW; ++j) {
    const int ml = j * 16 + r16;
    const int m = m0 + ml;
    float best = -INFINITY, mx = -INFINITY;
    int bidx = -1;
    if (m < p.M) {
#pragma unroll
      for (int i = 0; i < NBW; ++i) {
        const int nb = wave + 4 * i;
        if (nb >= nbtot) continue;
        const int n = nb * 16 + 4 * g;
        const float4 b4 = *reinterpret_cast<const float4*>(p.bc + n);
        const float lg[4] = {acc[i][j][0] + b4.x, acc[i][j][1] + b4.y, acc[i][j][2] + b4.z,
                             acc[i][j][3] + b4.w};
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          if (n + v == A) s_rho[ml][0] = lg[v];
          if (n + v == A + 1) s_rho[ml][1] = lg[v];
        }
        if (want_action && n < A) {
          const uint4 w = rng.block((uint32_t)(n >> 2), p.step, p.traj0 + (uint32_t)m, STREAM_CONTROLLER);
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            if ((mk[i][j] >> (8 * v)) & 1u) {
              mx = fmaxf(mx, lg[v]);
              const float s = lg[v] + gumbel(word_to_uniform(word_of(w, v)));
              if (s > best) { best = s; bidx = n + v; }
            }
          }
        }
      }
    }
    // reduce over the four lane groups (same row), lowest index on ties
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float ob = __shfl_xor(best, off);
      const int oi = __shfl_xor(bidx, off);
      const float om = __shfl_xor(mx, off);
      if (oi >= 0 && (bidx < 0 || ob > best || (ob == best && oi < bidx))) { best = ob; bidx = oi; }
      mx = fmaxf(mx, om);
    }
    if (g == 0) {
      s_best[wave][ml] = best;
      s_idx[wave][ml] = bidx;
      s_max[wave][ml] = mx;
    }
  }
  __syncthreads();

  if (p.mode == 0) {
    // combine waves; then probabilities
    if (tid < BM) {
      float best = -INFINITY, mx = -INFINITY;
      int bidx = -1;
      for (int w = 0; w < 4; ++w) {
        const float ob = s_best[w][tid];
        const int oi = s_idx[w][tid];
        if (oi >= 0 && (bidx < 0 || ob > best || (ob == best && oi < bidx))) { best = ob; bidx = oi; }
        mx = fmaxf(mx, s_max[w][tid]);
      }
      s_fin[tid][0] = mx;
      const int m = m0 + tid;
      if (m < p.M) p.action[m] = bidx;
    }
    __syncthreads();
    if (p.probs) {
      // sum of exp(l - max) over valid actions
#pragma unroll
      for (int j = 0; j < MBW; ++j) {
        const int ml = j * 16 + r16;
        const int m = m0 + ml;
        float se = 0.f;
        if (m < p.M) {
          const float mx = s_fin[ml][0];
#pragma unroll
          for (int i = 0; i < NBW; ++i) {
            const int nb = wave + 4 * i;
            if (nb >= nbtot) continue;
            const int n = nb * 16 + 4 * g;
#pragma unroll
            for (int v = 0; v < 4; ++v)
              if ((mk[i][j] >> (8 * v)) & 1u) se += expf(acc[i][j][v] + p.bc[n + v] - mx);
          }
        }
        se += __shfl_xor(se, 16);
        se += __shfl_xor(se, 32);
        if (g == 0) s_best[wave][ml] = se;
      }
      __syncthreads();
      if (tid < BM) s_fin[tid][1] = s_best[0][tid] + s_best[1][tid] + s_best[2][tid] + s_best[3][tid];
      __syncthreads();
#pragma unroll
      for (int j = 0; j < MBW; ++j) {
        const int ml = j * 16 + r16;
        const int m = m0 + ml;
        if (m >= p.M) continue;
        const float mx = s_fin[ml][0], inv = s_fin[ml][1] > 0.f ? 1.0f / s_fin[ml][1] : 0.f;
#pragma unroll
        for (int i = 0; i < NBW; ++i) {
          const int nb = wave + 4 * i;
          if (nb >= nbtot) continue;
          const int n = nb * 16 + 4 * g;
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            if (n + v < A) {
              const bool ok = (mk[i][j] >> (8 * v)) & 1u;
              p.probs[(long)m * A + n + v] = ok ? expf(acc[i][j][v] + p.bc[n + v] - mx) * inv : 0.f;
            }
          }
        }
      }
    }
    return;
  }

  // rollout modes: one thread per row
  if (tid < BM) {
    const int m = m0 + tid;
    if (m < p.M) {
      float best = -INFINITY;
      int a = -1;
      for (int w = 0; w < 4; ++w) {
        const float ob = s_best[w][tid];
        const int oi = s_idx[w][tid];
        if (oi >= 0 && (a < 0 || ob > best || (ob == best && oi < a))) { best = ob; a = oi; }
      }
      ctrl_row_commit(p, rng, m, a, s_rho[tid][0], s_rho[tid][1]);
    }
  }
}

// k_ctrl: controller on the pipelined GEMM core for A + 2 <= 64 * NBW
// outputs (all Nc weight rows of a row block in one tile).  The logit tile
// is staged through LDS as E[row][output]; each row is then handled by TPR
// adjacent threads, thread q taking the contiguous actions
// [q * APT, (q + 1) * APT) (APT a multiple of 4: one Philox block per four
// actions).  The mask bytes of those actions are fetched as 32-bit words
// before the GEMM when A % 4 == 0 (byte loads otherwise).
template <class C, class S>
__global__ void __launch_bounds__(C::NT) k_ctrl(const CtrlArgs p) {
  using DT = typename C::DT;
  constexpr int NBW = C::NBW, MBW = C::MBW, BM = C::BM;
  constexpr int TPR = C::NT / BM;               // threads per row
  constexpr int MAXB = (C::BN / TPR + 3) / 4;  // Philox blocks per thread
  constexpr int ELD = C::BN + 4;
  constexpr int E_BYTES = BM * ELD * 4;
  constexpr int LDS = C::LDS_BYTES > E_BYTES ? C::LDS_BYTES : E_BYTES;
  static_assert(C::NT % BM == 0 && (TPR & (TPR - 1)) == 0 && TPR <= 16, "row groups inside a wave");
  __shared__ __attribute__((aligned(16))) char lds_raw[LDS];

  const int m0 = blockIdx.x * BM;
  const int r = threadIdx.x / TPR, q = threadIdx.x % TPR;
  const int m = m0 + r;
  const bool row_ok = m < p.M;
  const int A = p.A;
  const int apt = (A + 4 * TPR - 1) / (4 * TPR) * 4;  // actions per thread
  const int a0 = q * apt;
  const bool want_action = p.mode != 2;

  // mask words of this thread's actions, ahead of the GEMM
  uint32_t mk[MAXB];
  const rsrc_t rmask = make_rsrc(p.mask + (long)m0 * A, (uint32_t)(max(0, min(BM, p.M - m0)) * A));
  const bool words = (A & 3) == 0 && (reinterpret_cast<uintptr_t>(p.mask) & 3) == 0;
#pragma unroll
  for (int b = 0; b < MAXB; ++b) {
    const int a = a0 + 4 * b;
    const bool ok = want_action && row_ok && p.N == 0 && 4 * b < apt && a < A;
    const uint32_t off = (uint32_t)(r * A + a);
    if (words) {
      mk[b] = bload4(rmask, ok ? off : kOffNone);
    } else {
      mk[b] = 0;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        mk[b] |= bload1(rmask, ok && a + v < A ? off + v : kOffNone) << (8 * v);
    }
  }

  const Rng rng{p.k0, p.k1};
  const uint32_t traj = p.traj0 + (uint32_t)m;
  const bool flat_pick = want_action && row_ok && p.N == 0;
  // On the sixteen-wave direct tile, the Gumbel noise of all of the thread's
  // actions is drawn while the GEMM's first chunks load (it does not depend
  // on the logits).  It is drawn whatever the mask: the mask words are still
  // in flight there, and waiting for them would wait for the chunks too.
  // (On the four-wave 32-row tiles of the large rollout the same draw made
  // the controller slower, 12.0 -> 12.8 us per step.)
  constexpr bool kPre = IsGemmD<C>::value && C::NT >= 1024 && MAXB <= 5;
  float gq[kPre ? MAXB : 1][4];
  auto draw = [&]() {
    if constexpr (kPre) {
#pragma unroll
      for (int b = 0; b < MAXB; ++b) {
        if (flat_pick && 4 * b < apt && a0 + 4 * b < A) {
          const uint4 wd = rng.block((uint32_t)((a0 + 4 * b) >> 2), p.step, traj, STREAM_CONTROLLER);
#pragma unroll
          for (int v = 0; v < 4; ++v) gq[b][v] = gumbel(word_to_uniform(word_of(wd, v)));
        }
      }
    }
  };

  f32x4 acc[NBW][MBW];
  const SrcX<DT> w(reinterpret_cast<const DT*>(p.Wc), p.ldk, p.ldk, 0, p.Nc, p.Nc);
  if constexpr (kPre)
    C::run(acc, w, ctrl_src<S>(p, m0, BM), (int)p.ldk, reinterpret_cast<DT*>(lds_raw), draw);
  else
    C::run(acc, w, ctrl_src<S>(p, m0, BM), (int)p.ldk, reinterpret_cast<DT*>(lds_raw));
  float* E = reinterpret_cast<float*>(lds_raw);
  if (C::kw() == 0) {
    const int lane = threadIdx.x & 63, r16 = lane & 15, g = lane >> 4;
    const int wn = C::wn(), wmi = C::wm();
#pragma unroll
    for (int j = 0; j < MBW; ++j)
#pragma unroll
      for (int i = 0; i < NBW; ++i)
        *reinterpret_cast<f32x4*>(E + ((wmi * MBW + j) * 16 + r16) * ELD + (wn * NBW + i) * 16 + 4 * g) =
            acc[i][j];
  }
  __syncthreads();

  const float* lg = E + r * ELD;
  float best = -INFINITY, mx = -INFINITY;
  int bidx = -1;
  if (flat_pick) {
#pragma unroll
    for (int b = 0; b < MAXB; ++b) {
      if (mk[b] == 0) continue;  // no valid action in the block (or outside the range)
      const int a = a0 + 4 * b;
      uint4 wd = make_uint4(0u, 0u, 0u, 0u);
      if constexpr (!kPre) wd = rng.block((uint32_t)(a >> 2), p.step, traj, STREAM_CONTROLLER);
      const float4 l4 = *reinterpret_cast<const float4*>(lg + a);
      const float4 b4 = *reinterpret_cast<const float4*>(p.bc + a);
      const float lv[4] = {l4.x + b4.x, l4.y + b4.y, l4.z + b4.z, l4.w + b4.w};
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        if ((mk[b] >> (8 * v)) & 0xffu) {
          mx = fmaxf(mx, lv[v]);
          float gv;
          if constexpr (kPre) gv = gq[b][v];
          else gv = gumbel(word_to_uniform(word_of(wd, v)));
          const float sc = lv[v] + gv;
          if (sc > best) { best = sc; bidx = a + v; }
        }
      }
    }
  }
  // reduce over the TPR threads of the row, lowest index on ties
#pragma unroll
  for (int off = 1; off < TPR; off <<= 1) {
    const float ob = __shfl_xor(best, off);
    const int oi = __shfl_xor(bidx, off);
    const float om = __shfl_xor(mx, off);
    if (oi >= 0 && (bidx < 0 || ob > best || (ob == best && oi < bidx))) { best = ob; bidx = oi; }
    mx = fmaxf(mx, om);
  }
  if (p.mode == 0) {
    if (row_ok && q == 0) p.action[m] = bidx;
    if (p.probs) {
      float se = 0.f;
#pragma unroll
      for (int b = 0; b < MAXB; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if ((mk[b] >> (8 * v)) & 0xffu) se += expf(lg[a0 + 4 * b + v] + p.bc[a0 + 4 * b + v] - mx);
#pragma unroll
      for (int off = 1; off < TPR; off <<= 1) se += __shfl_xor(se, off);
      const float inv = se > 0.f ? 1.0f / se : 0.f;
      if (row_ok) {
#pragma unroll
        for (int b = 0; b < MAXB; ++b)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int a = a0 + 4 * b + v;
            if (4 * b + v < apt && a < A)
              p.probs[(long)m * A + a] = ((mk[b] >> (8 * v)) & 0xffu) ? expf(lg[a] + p.bc[a] - mx) * inv : 0.f;
          }
      }
    }
    return;
  }
  if (p.N > 0) bidx = two_level_pick<TPR>(p, rng, lg, m, want_action && row_ok, q, traj);
  const int Ar = p.N > 0 ? p.N + 1 + p.Lc : A;  // the reward and done logit rows
  if (row_ok && q == 0) ctrl_row_commit(p, rng, m, bidx, lg[Ar] + p.bc[Ar], lg[Ar + 1] + p.bc[Ar + 1]);
}

// ===========================================================================
// Register-direct split-K GEMM for calls with few rows.  Every wave takes a
// contiguous run of at most SMAX MFMA K slices and loads all of its operand
// fragments for the whole tile straight from global memory into registers in
// one round trip (no LDS staging, no barrier inside the K loop), then runs
// its MFMAs.  The per-wave partial tiles meet in LDS and are summed in a
// fixed wave order, so results are deterministic; the sum lands in
// E[m][n] (tile rows m, features n, fp32) for an epilogue with any thread
// mapping.  The block has nwaves = blockDim.x / 64 waves, chosen by the host
// so that ceil(K slices / nwaves) <= SMAX.
// ===========================================================================
template <typename DT_, int NBW_, int MBW_, int SMAX_, int MAXT_>
struct GemmRD {
  using DT = DT_;
  static constexpr int NBW = NBW_, MBW = MBW_, SMAX = SMAX_;
  static constexpr int MAXT = MAXT_;  // largest block the kernels are compiled for
  static constexpr int KSLICE = Mfma<DT>::KSLICE, VEC = DType<DT>::VEC;
  static constexpr int BN = 16 * NBW, BM = 16 * MBW;
  static constexpr int TILE = BN * BM;  // floats per partial tile
  static constexpr int ELD = BN + 4;    // row stride of E (floats)

  static size_t lds_bytes(int nwaves) {
    return (size_t)nwaves * TILE * 4 + (size_t)BM * ELD * 4;
  }
  __device__ static float* E(float* lds) { return lds + (blockDim.x >> 6) * TILE; }

  // w: weight rows n0 .. n0+BN-1; x: activation rows m0 .. m0+BM-1.
  template <class S>
  __device__ __forceinline__ static void run(float* lds, const SrcX<DT>& w, const S& x, int Kpad) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int nsl = (Kpad + KSLICE - 1) / KSLICE;
    const int per = (nsl + nw - 1) / nw;
    const int s0 = wave * per;
    typename SrcX<DT>::Row wo[NBW];
    typename S::Row xo[MBW];
#pragma unroll
    for (int i = 0; i < NBW; ++i) wo[i] = w.row(i * 16 + r16);
#pragma unroll
    for (int j = 0; j < MBW; ++j) xo[j] = x.row(j * 16 + r16);
    uint4 wf[NBW][SMAX], xf[MBW][SMAX];
#pragma unroll
    for (int s = 0; s < SMAX; ++s) {
      const int sl = s0 + s;
      if (s < per && sl < nsl) {
        const int kl = sl * KSLICE + g * VEC;  // first column of this lane's vector
#pragma unroll
        for (int i = 0; i < NBW; ++i) wf[i][s] = w.load(wo[i], kl, Kpad);
#pragma unroll
        for (int j = 0; j < MBW; ++j) xf[j][s] = x.load(xo[j], kl, Kpad);
      } else {
#pragma unroll
        for (int i = 0; i < NBW; ++i) wf[i][s] = make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int j = 0; j < MBW; ++j) xf[j][s] = make_uint4(0, 0, 0, 0);
      }
    }
    f32x4 acc[NBW][MBW];
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
      for (int j = 0; j < MBW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < SMAX; ++s) {
      if (s < per && s0 + s < nsl) {
#pragma unroll
        for (int i = 0; i < NBW; ++i)
#pragma unroll
          for (int j = 0; j < MBW; ++j) Mfma<DT>::step(acc[i][j], wf[i][s], xf[j][s]);
      }
    }
    float* P = lds + wave * TILE;
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
      for (int j = 0; j < MBW; ++j)
        *reinterpret_cast<f32x4*>(P + ((i * MBW + j) * 64 + lane) * 4) = acc[i][j];
    __syncthreads();
    float* Et = E(lds);
    for (int e = threadIdx.x; e < TILE; e += blockDim.x) {
      float sum = 0.f;
      for (int w2 = 0; w2 < nw; ++w2) sum += lds[w2 * TILE + e];
      const int v = e & 3, l = (e >> 2) & 63, ij = e >> 8;
      const int j = ij % MBW, i = ij / MBW;
      Et[(j * 16 + (l & 15)) * ELD + i * 16 + 4 * (l >> 4) + v] = sum;
    }
    __syncthreads();
  }
};

// Gates on the register-direct core: tiles of BN/4 hidden units x BM rows.
// Each of the first threads owns one (unit, row) of the epilogue and issues
// its loads before the GEMM.
template <class R>
__global__ void __launch_bounds__(R::MAXT) k_gates_rd(const GatesArgs p) {
  using DT = typename R::DT;
  extern __shared__ __attribute__((aligned(16))) float lds_dyn[];
  int nt, mt;
  if (!tile_of(p.map, nt, mt)) return;
  const int n0 = nt * R::BN, m0 = mt * R::BM;
  constexpr int UPT = R::BN / 4;  // hidden units per tile
  static_assert(UPT * R::BM <= 256, "one epilogue element per thread of the first four waves");
  const int t = threadIdx.x;
  const int ul = t % UPT, ml = t / UPT;
  const int m = m0 + ml, u = n0 / 4 + ul;
  const bool mine = t < UPT * R::BM;
  const bool ok = mine && m < p.M && u < p.H;
  const GateIO<DT> io(p, m0, R::BM);
  GateIn in{};
  if (mine) in = io.load(ml, u, ok ? p.act[m] : -1, ok);
  const SrcX<DT> w(reinterpret_cast<const DT*>(p.Wg), p.ldk, p.ldk, n0, R::BN, 4 * p.H);
  const SrcX<DT> x(reinterpret_cast<const DT*>(p.x_in), p.ldx, p.ldx, m0, R::BM, p.M);
  R::run(lds_dyn, w, x, (int)p.ldk);
  if (mine) {
    const float4 g4 = *reinterpret_cast<const float4*>(R::E(lds_dyn) + ml * R::ELD + 4 * ul);
    io.commit(ml, u, ok, in, g4.x, g4.y, g4.z, g4.w);
  }
}

// Rollout mixture head on the register-direct core: one group of four
// latent dims (16Q feature rows) x BM rows per tile.  Each of the first
// threads owns one (dim, row) and draws its noise before the GEMM.
template <class R>
__global__ void __launch_bounds__(R::MAXT) k_mdn_rd(const MdnArgs p) {
  using DT = typename R::DT;
  constexpr int Q = R::NBW;
  extern __shared__ __attribute__((aligned(16))) float lds_dyn[];
  int J, mt;
  if (!tile_of(p.map, J, mt)) return;
  const int n0 = J * R::BN, m0 = mt * R::BM;
  const int t = threadIdx.x;
  const int d = t & 3, ml = t >> 2;
  const int m = m0 + ml, j = 4 * J + d;
  const bool mine = t < 4 * R::BM && m < p.M && j < p.Z;
  const Rng rng{p.k0, p.k1};
  bool live = false;
  float zprev = 0.f;
  MdnNoise noise{};
  if (mine) {
    live = p.act[m] >= 0;
    if (live) noise = mdn_noise(p, rng, m, j, p.K);
    else zprev = p.z_prev[(long)m * p.Z + j];
  }
  const SrcX<DT> w(reinterpret_cast<const DT*>(p.Wm), p.ldh, p.ldh, n0, R::BN, p.Nm);
  const SrcX<DT> x(reinterpret_cast<const DT*>(p.x) + p.Z, p.ldx, p.ldx - p.Z, m0, R::BM, p.M);
  R::run(lds_dyn, w, x, (int)p.ldh);
  if (!mine) return;
  if (!live) {
    mdn_commit<DT>(p, m, j, zprev);
    return;
  }
  const float* E = R::E(lds_dyn);
  float feat[4 * Q];
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = 16 * q + 4 * d + v;
      feat[4 * q + v] = E[ml * R::ELD + r] + p.bm[n0 + r];
    }
  mdn_commit<DT>(p, m, j, mdn_pick<Q>(p, noise, feat, p.K));
}

// Controller on the register-direct core: all Nc outputs x 16 rows.  Each row
// is handled by 16 lanes of one wave (four waves, four rows per wave), each
// lane taking the action blocks sub + 16 h, h < 4 (four actions and one
// Philox block each); their Gumbel noise and mask bits are drawn before the
// GEMM.  Requires A <= 256.
template <class R, class S>
__global__ void __launch_bounds__(R::MAXT) k_ctrl_rd(const CtrlArgs p) {
  using DT = typename R::DT;
  extern __shared__ __attribute__((aligned(16))) float lds_dyn[];
  const int m0 = blockIdx.x * R::BM;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int ml = 4 * wave + (lane >> 4), sub = lane & 15;
  const int m = m0 + ml;
  const bool row_ok = wave < 4 && m < p.M;
  const int A = p.A;
  const Rng rng{p.k0, p.k1};
  float gn[16];
  unsigned valid = 0;
  if (row_ok && p.mode != 2) {
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const int b = sub + 16 * h;
      if (4 * b < A) {
        const uint4 w = rng.block((uint32_t)b, p.step, p.traj0 + (uint32_t)m, STREAM_CONTROLLER);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int a = 4 * b + v;
          gn[4 * h + v] = gumbel(word_to_uniform(word_of(w, v)));
          if (a < A && p.mask[(long)m * A + a]) valid |= 1u << (4 * h + v);
        }
      }
    }
  }
  const SrcX<DT> w(reinterpret_cast<const DT*>(p.Wc), p.ldk, p.ldk, 0, R::BN, p.Nc);
  R::run(lds_dyn, w, ctrl_src<S>(p, m0, R::BM), (int)p.ldk);
  if (wave >= 4) return;  // rows live in the first four waves; no barrier below
  const float* lg = R::E(lds_dyn) + ml * R::ELD;
  float best = -INFINITY, mx = -INFINITY;
  int bidx = -1;
#pragma unroll
  for (int h = 0; h < 4; ++h)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if (valid & (1u << (4 * h + v))) {
        const int a = 4 * (sub + 16 * h) + v;
        const float l = lg[a] + p.bc[a];
        mx = fmaxf(mx, l);
        const float sc = l + gn[4 * h + v];
        if (sc > best) { best = sc; bidx = a; }
      }
    }
  // reduce over the 16 lanes of the row, lowest index on ties
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) {
    const float ob = __shfl_xor(best, off);
    const int oi = __shfl_xor(bidx, off);
    const float om = __shfl_xor(mx, off);
    if (oi >= 0 && (bidx < 0 || ob > best || (ob == best && oi < bidx))) { best = ob; bidx = oi; }
    mx = fmaxf(mx, om);
  }
  if (p.mode == 0) {
    if (row_ok && sub == 0) p.action[m] = bidx;
    if (p.probs) {
      float se = 0.f;
      if (row_ok)
        for (int a = sub; a < A; a += 16)
          if (p.mask[(long)m * A + a]) se += expf(lg[a] + p.bc[a] - mx);
#pragma unroll
      for (int off = 8; off >= 1; off >>= 1) se += __shfl_xor(se, off);
      const float inv = se > 0.f ? 1.0f / se : 0.f;
      if (row_ok)
        for (int a = sub; a < A; a += 16)
          p.probs[(long)m * A + a] = p.mask[(long)m * A + a] ? expf(lg[a] + p.bc[a] - mx) * inv : 0.f;
    }
    return;
  }
  if (row_ok && sub == 0) ctrl_row_commit(p, rng, m, bidx, lg[A] + p.bc[A], lg[A + 1] + p.bc[A + 1]);
}

// ===========================================================================
// small element-wise kernels
// ===========================================================================
// X_0 = [q(z0) | q(h0) | 0], zero padding columns of X_1, z_out[0] = z0,
// c = c0, done state, traces of step 0.
template <typename DT>
__global__ void k_rollout_init(int B, int Z, int H, int ldx, const float* __restrict__ z0,
                               const float* __restrict__ h0, const float* __restrict__ c0,
                               const uint8_t* __restrict__ done_io, float* __restrict__ z_out,
                               DT* __restrict__ X0, DT* __restrict__ X1, float* __restrict__ c,
                               int32_t* __restrict__ done_state, float* __restrict__ h_trace,
                               float* __restrict__ c_trace, unsigned* __restrict__ sync,
                               unsigned preset_err) {
  const long stride = (long)gridDim.x * blockDim.x;
  const long i0 = (long)blockIdx.x * blockDim.x + threadIdx.x;
  for (long i = i0; i < kSyncWords; i += stride) sync[i] = i == kSyncErr ? preset_err : 0u;
  for (long i = i0; i < (long)B * ldx; i += stride) {
    const long b = i / ldx;
    const int col = (int)(i % ldx);
    float v = 0.f;
    if (col < Z) v = z0[b * Z + col];
    else if (col < Z + H) v = h0 ? h0[b * H + col - Z] : 0.f;
    DType<DT>::store(X0, i, v);
    if (col >= Z + H) DType<DT>::store(X1, i, 0.f);
  }
  for (long i = i0; i < (long)B * Z; i += stride) z_out[i] = z0[i];
  for (long i = i0; i < (long)B * H; i += stride) {
    const float cv = c0 ? c0[i] : 0.f;
    c[i] = cv;
    if (h_trace) {
      h_trace[i] = DType<DT>::round(h0 ? h0[i] : 0.f);
      c_trace[i] = cv;
    }
  }
  for (long i = i0; i < B; i += stride) done_state[i] = done_io ? (done_io[i] != 0) : 0;
}

template <typename DT>
__global__ void k_rollout_finish(int B, int Z, int H, int ldx, const DT* __restrict__ XT,
                                 const float* __restrict__ c, const int32_t* __restrict__ done_state,
                                 float* __restrict__ h_T, float* __restrict__ c_T,
                                 uint8_t* __restrict__ done_io) {
  const long stride = (long)gridDim.x * blockDim.x;
  const long i0 = (long)blockIdx.x * blockDim.x + threadIdx.x;
  for (long i = i0; i < (long)B * H; i += stride) {
    if (h_T) h_T[i] = DType<DT>::load(XT, (i / H) * ldx + Z + i % H);
    if (c_T) c_T[i] = c[i];
  }
  if (done_io)
    for (long i = i0; i < B; i += stride) done_io[i] = (uint8_t)done_state[i];
}

// Padding of variable-length rollouts: z_out[t+1, b, :] = 0 for t >= lengths[b].
__global__ void k_rollout_pad(int T, int B, int Z, const int32_t* __restrict__ lengths,
                              float* __restrict__ z_out) {
  const long stride = (long)gridDim.x * blockDim.x;
  const long n = (long)T * B * Z;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const long tb = i / Z;
    const int t = (int)(tb / B), b = (int)(tb % B);
    if (t >= lengths[b]) z_out[(long)B * Z + i] = 0.f;
  }
}

// X_t[:, 0:Z] = q(z_t) for t = 0..T, padding columns zero, h_0 = c_0 = 0.
template <typename DT>
__global__ void k_nll_init(int T, int B, int Z, int H, int ldx, const float* __restrict__ z,
                           DT* __restrict__ X, float* __restrict__ c, unsigned* __restrict__ sync,
                           unsigned preset_err) {
  const long stride = (long)gridDim.x * blockDim.x;
  const long i0 = (long)blockIdx.x * blockDim.x + threadIdx.x;
  for (long i = i0; i < kSyncWords; i += stride) sync[i] = i == kSyncErr ? preset_err : 0u;
  const int ncol = ldx - H;  // z columns, then padding columns
  for (long i = i0; i < (long)(T + 1) * B * ncol; i += stride) {
    const long r = i / ncol;
    const int cc = (int)(i % ncol);
    if (cc < Z) DType<DT>::store(X, r * ldx + cc, z[r * Z + cc]);
    else DType<DT>::store(X, r * ldx + H + cc, 0.f);
  }
  for (long i = i0; i < (long)B * H; i += stride) {
    DType<DT>::store(X, (i / H) * ldx + Z + i % H, 0.f);
    c[i] = 0.f;
  }
}

// Per (t, b): sum the dim-tile partials, reward SE and done BCE from the head
// logits, padding mask; one partial sum per block for the means.
__global__ void __launch_bounds__(256)
    k_nll_reduce(int T, int B, int ntd, const float* __restrict__ part,
                 const float* __restrict__ head, const float* __restrict__ rewards,
                 const uint8_t* __restrict__ dones, const int32_t* __restrict__ lengths,
                 float* __restrict__ loglik, float* __restrict__ reward_se,
                 float* __restrict__ done_bce, float* __restrict__ wgsum) {
  __shared__ float s[4][256];
  const long M = (long)T * B;
  const long m = (long)blockIdx.x * 256 + threadIdx.x;
  float ll = 0.f, se = 0.f, bce = 0.f, cnt = 0.f;
  if (m < M) {
    const int t = (int)(m / B), b = (int)(m % B);
    int len = lengths ? lengths[b] : T;
    len = len < 0 ? 0 : (len > T ? T : len);
    if (t < len) {
      for (int k = 0; k < ntd; ++k) ll += part[m * ntd + k];
      const float rr = head[2 * m], rd = head[2 * m + 1];
      const float dr = rr - rewards[m];
      se = dr * dr;
      bce = fmaxf(rd, 0.f) + log1pf(expf(-fabsf(rd))) - (dones[m] ? rd : 0.f);
      cnt = 1.f;
    }
    loglik[m] = ll;
    reward_se[m] = se;
    done_bce[m] = bce;
  }
  s[0][threadIdx.x] = ll;
  s[1][threadIdx.x] = se;
  s[2][threadIdx.x] = bce;
  s[3][threadIdx.x] = cnt;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w)
      for (int k = 0; k < 4; ++k) s[k][threadIdx.x] += s[k][threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x < 4) wgsum[(long)blockIdx.x * 4 + threadIdx.x] = s[threadIdx.x][0];
}

__global__ void __launch_bounds__(256)
    k_nll_means(int nwg, int Z, const float* __restrict__ wgsum, float* __restrict__ means) {
  __shared__ double s[4][256];
  double acc[4] = {0, 0, 0, 0};
  for (int i = threadIdx.x; i < nwg; i += 256)
    for (int k = 0; k < 4; ++k) acc[k] += wgsum[(long)i * 4 + k];
  for (int k = 0; k < 4; ++k) s[k][threadIdx.x] = acc[k];
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w)
      for (int k = 0; k < 4; ++k) s[k][threadIdx.x] += s[k][threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double n = s[3][0];
    means[0] = n > 0 ? (float)(-s[0][0] / (n * Z)) : 0.f;
    means[1] = n > 0 ? (float)(s[1][0] / n) : 0.f;
    means[2] = n > 0 ? (float)(s[2][0] / n) : 0.f;
  }
}

// ===========================================================================
// host-side launch logic
// ===========================================================================
namespace {

// Tile configurations by dtype and call size.  "Small" tiles serve calls
// with up to kSmallRows rows (latency-bound: many work-groups, deep
// prefetch, K split across waves); "Large" tiles serve the big batches
// (MFMA-bound: more reuse per LDS byte).
constexpr int kSmallRows = 2048;


template <typename DT> struct Cfgs;
template <> struct Cfgs<float> {
  using GatesSmall = Gemm<float, 2, 1, 2, 2, 1, 32, 4>;  // 64 x 32
  using GatesLarge = GemmD<float, 4, 2, 2, 2, 2>;  // 128 x 64
  using GatesXL = GatesLarge;
  template <int Q> using MdnXL = GemmD<float, Q, 1, 2, 2, 2>;
  static constexpr bool kXL = false;  // fp32 calls this large take the 128 x 64 tiles
  template <int Q> using MdnSmall = Gemm<float, Q, 1, 2, 1, 2, 32, 4>;  // 32Q x 16, K split 2
  template <int Q> using MdnLarge = GemmD<float, Q, 1, 2, 2, 2>;
  template <int NB> using CtrlLarge = Gemm<float, NB, 4, 4, 1, 1, 32, 3>;  // 64NB x 64
  template <int NB> using CtrlLargeX = GemmD<float, NB, 2, 4, 1, 3>;      // 64NB x 32
  template <int NB> using CtrlXL = CtrlLargeX<NB>;
  static constexpr int WIDE_BKC = 64;
};
template <> struct Cfgs<bf16_t> {
  using GatesSmall = Gemm<bf16_t, 2, 1, 2, 2, 1, 64, 4>;
  using GatesLarge = GemmD<bf16_t, 4, 4, 2, 2, 2>;  // 128 x 128
  template <int Q> using MdnSmall = Gemm<bf16_t, Q, 1, 2, 1, 2, 64, 4>;
  template <int Q> using MdnLarge = GemmD<bf16_t, Q, 2, 2, 2, 2>;
  // many-tile calls: 256 x 256 gate tiles and 32Q x 256 mixture tiles on
  // eight waves halve the L2 -> LDS bytes per MFMA of the 128-wide tiles
  using GatesXL = GemmD<bf16_t, 4, 8, 4, 2, 2>;
  // (odd Q: 32Q + 256 rows do not deal evenly to eight waves' DMA loads)
  template <int Q> using MdnXL = std::conditional_t<Q % 2 == 0, GemmD<bf16_t, Q, 4, 2, 4, 2>, MdnLarge<Q>>;
  static constexpr bool kXL = true;
  template <int NB> using CtrlLarge = Gemm<bf16_t, NB, 4, 4, 1, 1, 64, 2>;
  template <int NB> using CtrlLargeX = GemmD<bf16_t, NB, 2, 4, 1, 3>;
  // 64-row controller tiles, three stages: half the weight re-reads of the
  // 32-row tiles.  With five 64-output blocks (A up to 318) sixteen waves of
  // one 16-row block each, which hide more of the chunk loads' latency than
  // eight waves of two (xlarge controller 23.9 -> 22.6 us per step; four
  // waves of four blocks: 32 us)
  template <int NB> using CtrlXL = std::conditional_t<NB == 5, GemmD<bf16_t, NB, 1, 4, 4, 3>,
                                                      GemmD<bf16_t, NB, 2, 4, 2, 3>>;
  static constexpr int WIDE_BKC = 128;
};

// The 256-row tiles serve calls that still give every CU at least one tile.
constexpr long kXLTiles = 256;

// Register-direct kernels serve calls with at most this many rows, when the
// K slices fit SMAX per wave on the compiled block size.
constexpr int kRdGatesRows = 256, kRdMdnRows = 1024, kRdCtrlRows = 1024;
constexpr size_t kRdLdsMax = 64 * 1024;

inline int rd_waves(int Kpad, int kslice, int smax, int min_waves) {
  const int nsl = (Kpad + kslice - 1) / kslice;
  int nw = (nsl + smax - 1) / smax;
  return nw < min_waves ? min_waves : nw;
}

// Dynamic LDS above the default needs the kernel attribute raised once.
template <typename F>
hipError_t allow_lds(F* kernel, size_t bytes) {
  if (bytes <= 64 * 1024) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

// Weight bytes an XCD should keep in its L2 (4 MB) while activations stream.
constexpr size_t kL2Budget = 2560 * 1024;

// Picks gn for nt x mt tiles over `wbytes` of weights: the weights' per-XCD
// slice fits the L2 budget if possible, then the busiest XCD gets the fewest
// tiles, then the activations are re-read by the fewest XCD groups.
TileMap tile_map(int nt, int mt, size_t wbytes) {
  TileMap best{};
  bool best_fits = false;
  long best_tiles = 0;
  for (int gn = 1; gn <= 8; gn *= 2) {
    if (gn > 1 && gn > nt) break;
    TileMap t{nt, mt, gn, (nt + gn - 1) / gn, (mt + 8 / gn - 1) / (8 / gn)};
    const bool fits = wbytes / gn <= kL2Budget;
    const long tiles = (long)t.nper * t.mper;
    if (gn == 1 || (fits && !best_fits) || (fits == best_fits && tiles < best_tiles)) {
      best = t;
      best_fits = fits;
      best_tiles = tiles;
    }
  }
  return best;
}

unsigned grid_of(const TileMap& t) { return (unsigned)(8 * t.nper * t.mper); }

template <class C, typename DT>
hipError_t launch_gates_cfg(GatesArgs a, hipStream_t s) {
  a.map = tile_map((4 * a.H + C::BN - 1) / C::BN, (a.M + C::BM - 1) / C::BM,
                   (size_t)4 * a.H * a.ldk * sizeof(DT));
  return launch("gates", k_gates<C>, dim3(grid_of(a.map)), dim3(C::NT), 0, s, a);
}

// Register-direct gate launch with tile R; returns hipErrorNotSupported
// when the K slices do not fit the compiled block size or the LDS budget.
template <class R, typename DT>
hipError_t launch_gates_rd(GatesArgs a, hipStream_t s) {
  const int nw = rd_waves((int)a.ldk, R::KSLICE, R::SMAX, 4);
  const size_t lds = R::lds_bytes(nw);
  if (64 * nw > R::MAXT || lds > kRdLdsMax) return hipErrorNotSupported;
  hipError_t e = allow_lds(k_gates_rd<R>, lds);
  if (e != hipSuccess) return e;
  a.map = tile_map((4 * a.H + R::BN - 1) / R::BN, (a.M + R::BM - 1) / R::BM,
                   (size_t)4 * a.H * a.ldk * sizeof(DT));
  return launch("gates", k_gates_rd<R>, dim3(grid_of(a.map)), dim3(64 * nw), lds, s, a);
}

template <typename DT>
hipError_t launch_gates(GatesArgs a, hipStream_t s) {
  if (a.M <= kRdGatesRows) {
    // 16-row tiles for a single row block, 32-row tiles above
    const hipError_t e = a.M <= 16 ? launch_gates_rd<GemmRD<DT, 2, 1, 4, 640>, DT>(a, s)
                                   : launch_gates_rd<GemmRD<DT, 2, 2, 4, 640>, DT>(a, s);
    if (e != hipErrorNotSupported) return e;
  }
  if (a.M <= kSmallRows) return launch_gates_cfg<typename Cfgs<DT>::GatesSmall, DT>(a, s);
  using XL = typename Cfgs<DT>::GatesXL;
  if (Cfgs<DT>::kXL && (long)((4 * a.H + XL::BN - 1) / XL::BN) * ((a.M + XL::BM - 1) / XL::BM) >= kXLTiles) {
    if constexpr (sizeof(DT) == 2 && XL::NBW == 4 && XL::KSPLIT == 1) {
      a.map = tile_map((4 * a.H + XL::BN - 1) / XL::BN, (a.M + XL::BM - 1) / XL::BM,
                       (size_t)4 * a.H * a.ldk * sizeof(DT));
      return launch("gates", k_gates_direct<XL>, dim3(grid_of(a.map)), dim3(XL::NT), 0, s, a);
    } else {
      return launch_gates_cfg<XL, DT>(a, s);
    }
  }
  return launch_gates_cfg<typename Cfgs<DT>::GatesLarge, DT>(a, s);
}

template <class C, typename DT, int KC>
hipError_t launch_mdn_cfg(MdnArgs a, int ntiles, hipStream_t s) {
  a.map = tile_map(ntiles, (a.M + C::BM - 1) / C::BM, (size_t)a.Nm * a.ldh * sizeof(DT));
  return launch("mdn", k_mdn<C, KC>, dim3(grid_of(a.map)), dim3(C::NT), 0, s, a);
}

template <typename DT, int Q, int KC>
hipError_t launch_mdn_q(const MdnArgs& a, int ntiles, hipStream_t s) {
  if (!a.nll_mode) {
    using R = GemmRD<DT, Q, 1, 4, 640>;  // 16-row tiles: more work-groups
    const int nw = rd_waves((int)a.ldh, R::KSLICE, R::SMAX, 4);
    const size_t lds = R::lds_bytes(nw);
    if (a.M <= kRdMdnRows && 64 * nw <= R::MAXT && lds <= kRdLdsMax) {
      hipError_t e = allow_lds(k_mdn_rd<R>, lds);
      if (e != hipSuccess) return e;
      MdnArgs b = a;
      // one dim group per tile
      b.map = tile_map(a.Z / 4, (a.M + R::BM - 1) / R::BM, (size_t)a.Nm * a.ldh * sizeof(DT));
      return launch("mdn", k_mdn_rd<R>, dim3(grid_of(b.map)), dim3(64 * nw), lds, s, b);
    }
  }
  if (a.M <= kSmallRows) return launch_mdn_cfg<typename Cfgs<DT>::template MdnSmall<Q>, DT, KC>(a, ntiles, s);
  using XL = typename Cfgs<DT>::template MdnXL<Q>;
  if (Cfgs<DT>::kXL && (long)ntiles * ((a.M + XL::BM - 1) / XL::BM) >= kXLTiles)
    return launch_mdn_cfg<XL, DT, KC>(a, ntiles, s);
  return launch_mdn_cfg<typename Cfgs<DT>::template MdnLarge<Q>, DT, KC>(a, ntiles, s);
}

// one instantiation per component count K (which fixes Q = ceil(3K / 4))
template <typename DT>
hipError_t launch_mdn(const MdnArgs& a, int Q, int ntiles, hipStream_t s) {
  if (a.K < 1 || a.K > 8 || Q != (3 * a.K + 3) / 4) return hipErrorInvalidValue;
  switch (a.K) {
    case 1: return launch_mdn_q<DT, 1, 1>(a, ntiles, s);
    case 2: return launch_mdn_q<DT, 2, 2>(a, ntiles, s);
    case 3: return launch_mdn_q<DT, 3, 3>(a, ntiles, s);
    case 4: return launch_mdn_q<DT, 3, 4>(a, ntiles, s);
    case 5: return launch_mdn_q<DT, 4, 5>(a, ntiles, s);
    case 6: return launch_mdn_q<DT, 5, 6>(a, ntiles, s);
    case 7: return launch_mdn_q<DT, 6, 7>(a, ntiles, s);
    default: return launch_mdn_q<DT, 6, 8>(a, ntiles, s);
  }
}

template <class C, class S>
hipError_t launch_ctrl_cfg(const CtrlArgs& a, hipStream_t s) {
  return launch("ctrl", k_ctrl<C, S>, dim3((a.M + C::BM - 1) / C::BM), dim3(C::NT), 0, s, a);
}

template <class S, int NBW, int MBW>
hipError_t launch_ctrl_wide(const CtrlArgs& a, hipStream_t s) {
  constexpr int BM = 16 * MBW;
  return launch("ctrl", k_ctrl_wide<S, NBW, MBW, Cfgs<typename S::DT>::WIDE_BKC>,
                dim3((a.M + BM - 1) / BM), dim3(256), 0, s, a);
}

template <class R, class S>
hipError_t launch_ctrl_rd(const CtrlArgs& a, int nw, hipStream_t s) {
  const size_t lds = R::lds_bytes(nw);
  hipError_t e = allow_lds(k_ctrl_rd<R, S>, lds);
  if (e != hipSuccess) return e;
  return launch("ctrl", k_ctrl_rd<R, S>, dim3((a.M + R::BM - 1) / R::BM), dim3(64 * nw), lds, s, a);
}

// S: activation source (SrcX for the rollout's X_t, SrcZH for the step).
template <class S>
hipError_t launch_ctrl(const CtrlArgs& a, hipStream_t s) {
  using DT = typename S::DT;
  using Cf = Cfgs<DT>;
  const int nbtot = a.Nc / 16;
  const int nbw = (nbtot + 3) / 4;  // output blocks per wave over four waves
  // the two-level controller of the controller step, and in rollouts where
  // its logit rows do not fit the staged tiles: the logits are stored (into
  // probs for the step, the workspace in a rollout), then picked per row
  if (a.N > 0 && (a.mode == 0 || nbw > 5)) {
    CtrlArgs g = a;
    g.logits_out = a.mode == 0 ? a.probs : a.lg_ws;
    g.ldl = a.mode == 0 ? a.N + 1 + a.Lc : a.Nc;
    g.ncol = a.mode == 0 ? a.N + 1 + a.Lc : a.Nc;
    if (!g.logits_out) return hipErrorInvalidValue;
    hipError_t e;
    if (nbw <= 8) e = launch_ctrl_wide<S, 8, 2>(g, s);
    else if (nbw <= 12) e = launch_ctrl_wide<S, 12, 2>(g, s);
    else if (nbw <= 17) e = launch_ctrl_wide<S, 17, 1>(g, s);
    else if (nbw <= 24) e = launch_ctrl_wide<S, 24, 1>(g, s);
    else if (nbw <= 33) e = launch_ctrl_wide<S, 33, 1>(g, s);
    else return hipErrorInvalidValue;
    if (e != hipSuccess) return e;
    return launch("ctrl", k_ctrl_rows, dim3((unsigned)((a.M + 3) / 4)), dim3(256), 0, s, g);
  }
  // (otherwise the two-level controller runs on the kernels that stage whole logit rows)
  if (a.M <= kRdCtrlRows && nbtot <= 9 && a.N == 0) {
    const int nb = nbtot <= 1 ? 1 : nbtot <= 2 ? 2 : nbtot <= 3 ? 3 : nbtot <= 5 ? 5 : 9;
    const int smax = nb <= 5 ? 8 : 4;  // register budget
    const int nw = rd_waves((int)a.ldk, Mfma<DT>::KSLICE, smax, 4);
    if (nw <= 8 && GemmRD<DT, 9, 1, 4, 512>::lds_bytes(nw) <= kRdLdsMax) {
      switch (nb) {
        case 1: return launch_ctrl_rd<GemmRD<DT, 1, 1, 8, 512>, S>(a, nw, s);
        case 2: return launch_ctrl_rd<GemmRD<DT, 2, 1, 8, 512>, S>(a, nw, s);
        case 3: return launch_ctrl_rd<GemmRD<DT, 3, 1, 8, 512>, S>(a, nw, s);
        case 5: return launch_ctrl_rd<GemmRD<DT, 5, 1, 8, 512>, S>(a, nw, s);
        default: return launch_ctrl_rd<GemmRD<DT, 9, 1, 4, 512>, S>(a, nw, s);
      }
    }
  }
  const int nb = nbw;
  if constexpr (S::kTwo) {
    if (nb <= 1) return launch_ctrl_cfg<typename Cf::template CtrlLarge<1>, S>(a, s);
    if (nb <= 2) return launch_ctrl_cfg<typename Cf::template CtrlLarge<2>, S>(a, s);
    if (nb <= 3) return launch_ctrl_cfg<typename Cf::template CtrlLarge<3>, S>(a, s);
    if (nb <= 5) return launch_ctrl_cfg<typename Cf::template CtrlLarge<5>, S>(a, s);
  } else {
    // 64-row tiles once they still give every CU one, 32-row tiles below
    if (Cf::kXL && (long)(a.M + 63) / 64 >= kXLTiles) {
      if (nb <= 1) return launch_ctrl_cfg<typename Cf::template CtrlXL<1>, S>(a, s);
      if (nb <= 2) return launch_ctrl_cfg<typename Cf::template CtrlXL<2>, S>(a, s);
      if (nb <= 3) return launch_ctrl_cfg<typename Cf::template CtrlXL<3>, S>(a, s);
      if (nb <= 5) return launch_ctrl_cfg<typename Cf::template CtrlXL<5>, S>(a, s);
    }
    if (nb <= 1) return launch_ctrl_cfg<typename Cf::template CtrlLargeX<1>, S>(a, s);
    if (nb <= 2) return launch_ctrl_cfg<typename Cf::template CtrlLargeX<2>, S>(a, s);
    if (nb <= 3) return launch_ctrl_cfg<typename Cf::template CtrlLargeX<3>, S>(a, s);
    if (nb <= 5) return launch_ctrl_cfg<typename Cf::template CtrlLargeX<5>, S>(a, s);
  }
  if (nb <= 8) return launch_ctrl_wide<S, 8, 2>(a, s);
  if (nb <= 12) return launch_ctrl_wide<S, 12, 2>(a, s);
  if (nb <= 17) return launch_ctrl_wide<S, 17, 1>(a, s);
  if (nb <= 24) return launch_ctrl_wide<S, 24, 1>(a, s);
  if (nb <= 33) return launch_ctrl_wide<S, 33, 1>(a, s);
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// WM_FLAG_CHECK: device-side precondition checks.  Each thread counts the
// violations in its grid-stride share and adds a nonzero count to the
// status word sync[kSyncViol]; k_check_zero first clears both status words
// (the workspace's bytes are the caller's until the call's init kernel).
// ---------------------------------------------------------------------------
__global__ void k_check_zero(unsigned* __restrict__ sync) {
  if (threadIdx.x == 0) {
    sync[kSyncErr] = 0u;
    sync[kSyncViol] = 0u;
  }
}

// bytes other than 0 and 1 (the masks)
__global__ void k_check_bytes01(const uint8_t* __restrict__ p, long n, unsigned* __restrict__ sync) {
  const long stride = (long)gridDim.x * blockDim.x;
  unsigned bad = 0;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) bad += p[i] > 1u;
  if (bad) atomicAdd(sync + kSyncViol, bad);
}

// steps inside their sequence (t < lengths[b]): an action outside
// [0, A) u {-1, -2}, or a done byte other than 0 and 1
__global__ void k_check_nll(int T, int B, int A, const int32_t* __restrict__ actions,
                            const uint8_t* __restrict__ dones, const int32_t* __restrict__ lengths,
                            unsigned* __restrict__ sync) {
  const long stride = (long)gridDim.x * blockDim.x;
  unsigned bad = 0;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < (long)T * B; i += stride) {
    const int t = (int)(i / B), b = (int)(i % B);
    if (lengths && t >= lengths[b]) continue;
    const int32_t a = actions[i];
    bad += (a >= A || a < -2) + (dones[i] > 1u);
  }
  if (bad) atomicAdd(sync + kSyncViol, bad);
}

unsigned elem_grid(long n) {
  long g = (n + 255) / 256;
  if (g < 1) g = 1;
  if (g > 4096) g = 4096;
  return (unsigned)g;
}

// After the last step: the final state and done flags, and the padding of
// variable-length rollouts.
template <typename DT>
hipError_t rollout_tail(const Layout& L, const RolloutBufs& R, const DT* XT, hipStream_t s) {
  const long BH = (long)R.B * L.H;
  hipError_t e = launch("finish", k_rollout_finish<DT>, dim3(elem_grid(BH)), dim3(256), 0, s, R.B, L.Z, L.H,
                        L.ldx, XT, R.c, R.done_state, R.h_T, R.c_T, R.done_io);
  if (e != hipSuccess || !R.lengths) return e;
  return launch("finish", k_rollout_pad, dim3(elem_grid((long)R.T * R.B * L.Z)), dim3(256), 0, s, R.T, R.B,
                L.Z, R.lengths, R.z_out);
}

template <typename DT>
hipError_t rollout_impl(const Packed& P, const RolloutBufs& R, hipStream_t s) {
  const Layout& L = P.L;
  const char* base = reinterpret_cast<const char*>(P.base);
  const int B = R.B, T = R.T, Z = L.Z, H = L.H;
  DT* X = reinterpret_cast<DT*>(R.x);
  const long BX = (long)B * L.ldx, BH = (long)B * H, BZ = (long)B * Z;
  const bool trace = (R.flags & WM_FLAG_TRACE) != 0;
  hipError_t e = launch("init", k_rollout_init<DT>, dim3(elem_grid(BX)), dim3(256), 0, s, B, Z, H,
                        L.ldx, R.z0, R.h0, R.c0, R.done_io, R.z_out, X, X + BX, R.c, R.done_state,
                        trace ? R.h_trace : nullptr, trace ? R.c_trace : nullptr, R.sync,
                        R.preset_err);
  if (e != hipSuccess) return e;
  if (T > 0) {
    // one persistent launch for every step when the batch and dims allow it
    e = launch_rollout_persist(P, R, s);
    if (e == hipSuccess) return rollout_tail<DT>(L, R, X + (long)(T & 1) * BX, s);
    if (e != hipErrorNotSupported) return e;
  }

  CtrlArgs ca{};
  ca.Wc = base + L.off_Wc;
  ca.bc = reinterpret_cast<const float*>(base + L.off_bc);
  ca.ldk = L.ldk;
  ca.Z = Z; ca.H = H; ca.A = L.A; ca.Nc = L.Nc; ca.M = B;
  ca.ldx = L.ldx;
  ca.mask = R.mask;
  ca.k0 = R.k0; ca.k1 = R.k1; ca.traj0 = R.traj0;
  ca.done_state = R.done_state;
  ca.use_done = (R.flags & WM_FLAG_DONE) != 0;
  ca.lengths = R.lengths;
  ca.lg_ws = R.lg;
  ca.N = L.N;
  ca.Lc = L.Lc;

  GatesArgs ga{};
  ga.Wg = base + L.off_Wg;
  ga.WaT = base + L.off_WaT;
  ga.bg = reinterpret_cast<const float*>(base + L.off_bg);
  ga.ldk = L.ldk;
  ga.ldx = L.ldx;
  ga.H = H; ga.A = L.A; ga.Z = Z; ga.M = B;
  ga.nll_mode = 0;
  ga.c = R.c;

  MdnArgs ma{};
  ma.Wm = base + L.off_Wm;
  ma.bm = reinterpret_cast<const float*>(base + L.off_bm);
  ma.ldh = L.ldh;
  ma.ldx = L.ldx;
  ma.H = H; ma.Z = Z; ma.K = L.K; ma.Nm = L.Nm; ma.M = B;
  ma.k0 = R.k0; ma.k1 = R.k1; ma.traj0 = R.traj0; ma.tau = R.tau;
  ma.sig = (R.flags & WM_FLAG_SIGMA_TAU) ? sqrtf(R.tau) : 1.0f;
  ma.nll_mode = 0;
  const int mdn_tiles = Z / 8;

  for (int t = 0; t <= T; ++t) {
    const uint32_t step = R.step0 + (uint32_t)t;
    DT* Xt = X + (long)(t & 1) * BX;
    DT* Xn = X + (long)((t + 1) & 1) * BX;
    ca.x = Xt;
    ca.step = step;
    ca.t = t;
    ca.mode = t < T ? 1 : 2;
    // step t's [B, A] slice of a per-step mask (the tail step draws no action)
    ca.mask = (R.flags & WM_FLAG_STEP_MASK) ? R.mask + (long)(t < T ? t : T - 1) * B * L.A : R.mask;
    ca.act_t = t < T ? R.actions + (long)t * B : nullptr;
    ca.rew_t = t < T ? R.rewards + (long)t * B : nullptr;
    ca.done_t = t < T ? R.dones + (long)t * B : nullptr;
    ca.act_prev = t > 0 ? R.actions + (long)(t - 1) * B : nullptr;
    ca.rew_prev = t > 0 ? R.rewards + (long)(t - 1) * B : nullptr;
    ca.done_prev = t > 0 ? R.dones + (long)(t - 1) * B : nullptr;
    e = launch_ctrl<SrcX<DT>>(ca, s);
    if (e != hipSuccess) return e;
    if (t == T) break;

    ga.x_in = Xt;
    ga.x_out = Xn;
    ga.act = R.actions + (long)t * B;
    ga.h_trace = trace ? R.h_trace + (long)(t + 1) * BH : nullptr;
    ga.c_trace = trace ? R.c_trace + (long)(t + 1) * BH : nullptr;
    e = launch_gates<DT>(ga, s);
    if (e != hipSuccess) return e;

    ma.x = Xn;
    ma.act = R.actions + (long)t * B;
    ma.z_prev = R.z_out + (long)t * BZ;
    ma.z_next = R.z_out + (long)(t + 1) * BZ;
    ma.step = step;
    e = launch_mdn<DT>(ma, L.Q, mdn_tiles, s);
    if (e != hipSuccess) return e;
  }
  return rollout_tail<DT>(L, R, X + (long)(T & 1) * BX, s);
}

// heads = false: the recurrence only (X_1 .. X_T), for the training gradient
template <typename DT>
hipError_t nll_impl(const Packed& P, const NllBufs& N, hipStream_t s, bool heads = true) {
  const Layout& L = P.L;
  const char* base = reinterpret_cast<const char*>(P.base);
  const int B = N.B, T = N.T, Z = L.Z, H = L.H;
  const long BX = (long)B * L.ldx, BZ = (long)B * Z, M = (long)T * B;
  DT* X = reinterpret_cast<DT*>(N.x);
  hipError_t e = launch("nll_init", k_nll_init<DT>, dim3(elem_grid((long)(T + 1) * B * (L.ldx - H))),
                        dim3(256), 0, s, T, B, Z, H, L.ldx, N.z, X, N.c, N.sync, N.preset_err);
  if (e != hipSuccess) return e;

  GatesArgs ga{};
  ga.Wg = base + L.off_Wg;
  ga.WaT = base + L.off_WaT;
  ga.bg = reinterpret_cast<const float*>(base + L.off_bg);
  ga.ldk = L.ldk;
  ga.ldx = L.ldx;
  ga.H = H; ga.A = L.A; ga.Z = Z; ga.M = B;
  ga.nll_mode = 1;
  ga.c = N.c;
  // the recurrence: one persistent launch when the batch and dims allow it
  e = launch_nll_persist(P, N, s);
  if (e != hipSuccess && e != hipErrorNotSupported) return e;
  for (int t = 0; e == hipErrorNotSupported && t < T; ++t) {
    ga.x_in = X + (long)t * BX;
    ga.x_out = X + (long)(t + 1) * BX;
    ga.act = N.actions + (long)t * B;
    const hipError_t eg = launch_gates<DT>(ga, s);
    if (eg != hipSuccess) return eg;
  }
  if (!heads) return hipSuccess;

  const int ntd = Z / 8;
  MdnArgs ma{};
  ma.Wm = base + L.off_Wm;
  ma.bm = reinterpret_cast<const float*>(base + L.off_bm);
  ma.ldh = L.ldh;
  ma.ldx = L.ldx;
  ma.H = H; ma.Z = Z; ma.K = L.K; ma.Nm = L.Nm; ma.M = (int)M;
  ma.x = X + BX;  // rows of X_1 .. X_T
  ma.z_tgt = N.z + BZ;
  ma.part = N.part;
  ma.head = N.head;
  ma.ntd = ntd;
  ma.nll_mode = 1;
  e = launch_mdn<DT>(ma, L.Q, ntd + 1, s);
  if (e != hipSuccess) return e;

  const int nwg = (int)((M + 255) / 256);
  e = launch("nll_reduce", k_nll_reduce, dim3(nwg), dim3(256), 0, s, T, B, ntd, N.part, N.head,
             N.rewards, N.dones, N.lengths, N.loglik, N.reward_se, N.done_bce, N.wgsum);
  if (e != hipSuccess || !N.means) return e;
  return launch("nll_means", k_nll_means, dim3(1), dim3(256), 0, s, nwg, Z, N.wgsum, N.means);
}

}  // namespace

size_t rollout_workspace(const Layout& L, int B, char* ws, RolloutBufs* R) {
  size_t o = 0;
  const size_t os = o;
  o = wm_align256(o + (size_t)kSyncWords * 4);  // barrier and status words
  const size_t ox = o;
  o = wm_align256(o + (size_t)2 * B * L.ldx * L.esz);  // X_t, X_t+1
  const size_t oc = o;
  o = wm_align256(o + (size_t)B * L.H * 4);  // c
  const size_t od = o;
  o = wm_align256(o + (size_t)B * 4);  // done state
  const size_t pb = persist_partial_bytes(L, B);
  const size_t op = o;
  o = wm_align256(o + pb);  // persistent-kernel controller partials
  // logits of a two-level controller too wide for the staged tiles
  const bool wide2 = L.N > 0 && (L.Nc / 16 + 3) / 4 > 5;
  const size_t og = o;
  if (wide2) o = wm_align256(o + (size_t)B * L.Nc * 4);
  if (ws && R) {
    R->lg = wide2 ? reinterpret_cast<float*>(ws + og) : nullptr;
    R->x = ws + ox;
    R->c = reinterpret_cast<float*>(ws + oc);
    R->done_state = reinterpret_cast<int32_t*>(ws + od);
    R->sync = reinterpret_cast<unsigned*>(ws + os);
    R->P = pb ? reinterpret_cast<float*>(ws + op) : nullptr;
  }
  return o;
}

size_t nll_workspace(const Layout& L, int B, int T, char* ws, NllBufs* N) {
  const size_t M = (size_t)T * B;
  size_t o = 0;
  const size_t os = o;
  o = wm_align256(o + (size_t)kSyncWords * 4);  // barrier and status words
  const size_t ox = o;
  o = wm_align256(o + (size_t)(T + 1) * B * L.ldx * L.esz);  // X_0 .. X_T
  const size_t oc = o;
  o = wm_align256(o + (size_t)B * L.H * 4);  // c
  const size_t op = o;
  o = wm_align256(o + M * (L.Z / 8) * 4);  // dim-tile partials
  const size_t oh = o;
  o = wm_align256(o + M * 2 * 4);  // reward / done logits
  const size_t og = o;
  o = wm_align256(o + ((M + 255) / 256) * 4 * 4);  // block sums
  if (ws && N) {
    N->sync = reinterpret_cast<unsigned*>(ws + os);
    N->x = ws + ox;
    N->c = reinterpret_cast<float*>(ws + oc);
    N->part = reinterpret_cast<float*>(ws + op);
    N->head = reinterpret_cast<float*>(ws + oh);
    N->wgsum = reinterpret_cast<float*>(ws + og);
  }
  return o;
}

hipError_t launch_check_zero(unsigned* sync, hipStream_t s) {
  return launch("check", k_check_zero, dim3(1), dim3(64), 0, s, sync);
}

hipError_t launch_check_bytes01(const uint8_t* p, long n, unsigned* sync, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  return launch("check", k_check_bytes01, dim3(elem_grid(n)), dim3(256), 0, s, p, n, sync);
}

hipError_t launch_check_nll(int T, int B, int A, const int32_t* actions, const uint8_t* dones,
                            const int32_t* lengths, unsigned* sync, hipStream_t s) {
  if ((long)T * B <= 0) return hipSuccess;
  return launch("check", k_check_nll, dim3(elem_grid((long)T * B)), dim3(256), 0, s, T, B, A, actions,
                dones, lengths, sync);
}

hipError_t launch_pack(const Packed& P, void* packed, const float* W_g, const float* b_g,
                       const float* W_m, const float* b_m, const float* w_r, const float* b_r,
                       const float* w_d, const float* b_d, const float* W_c, const float* b_c,
                       hipStream_t s) {
  char* out = reinterpret_cast<char*>(packed);
  if (P.L.dt == 0)  // two more sections: the transposed copies
    return launch("pack", k_pack<float>, dim3(1024, 9), dim3(256), 0, s, P.L, out, W_g, b_g, W_m, b_m, w_r,
                  b_r, w_d, b_d, W_c, b_c);
  return launch("pack", k_pack<bf16_t>, dim3(1024, 7), dim3(256), 0, s, P.L, out, W_g, b_g, W_m, b_m, w_r, b_r,
                w_d, b_d, W_c, b_c);
}

hipError_t launch_controller_step(const Packed& P, int B, uint32_t traj0, const float* z,
                                  const float* h, const uint8_t* mask, uint32_t k0, uint32_t k1,
                                  uint32_t step, float* probs, int32_t* action, hipStream_t s) {
  const Layout& L = P.L;
  const char* base = reinterpret_cast<const char*>(P.base);
  CtrlArgs ca{};
  ca.Wc = base + L.off_Wc;
  ca.bc = reinterpret_cast<const float*>(base + L.off_bc);
  ca.ldk = L.ldk;
  ca.Z = L.Z; ca.H = L.H; ca.A = L.A; ca.Nc = L.Nc; ca.M = B;
  ca.z = z;
  ca.h = h;
  ca.mask = mask;
  ca.k0 = k0; ca.k1 = k1; ca.step = step; ca.traj0 = traj0;
  ca.mode = 0;
  ca.probs = probs;
  ca.action = action;
  ca.N = L.N;
  ca.Lc = L.Lc;
  if (L.dt == 0) return launch_ctrl<SrcZH<float>>(ca, s);
  return launch_ctrl<SrcZH<bf16_t>>(ca, s);
}

hipError_t launch_rollout(const Packed& P, const RolloutBufs& R, hipStream_t s) {
  return P.L.dt == 0 ? rollout_impl<float>(P, R, s) : rollout_impl<bf16_t>(P, R, s);
}

hipError_t launch_nll(const Packed& P, const NllBufs& N, hipStream_t s) {
  return P.L.dt == 0 ? nll_impl<float>(P, N, s) : nll_impl<bf16_t>(P, N, s);
}

// ===========================================================================
// World-model training step: the gradient of the summed NLL means with
// respect to the gate, mixture, reward and done weights (fp32), by
// backpropagation through time after the forward NLL pass.
//
//   forward   X (z_t | h_t) from the NLL pass; where the persistent kernel
//             runs it, the gate activations and c_{t+1} of every step come
//             with it; otherwise the pre-activations of every step in one
//             GEMM and a scan that adds bias and one-hot column, applies the
//             gates and records c_t
//   heads     mixture/reward/done outputs of every h_{t+1} in one GEMM; an
//             element-wise kernel turns them into d loss / d output (dM)
//   back      dh_heads = dM W_m; per step (backwards) the LSTM backward gives
//             dG_t and dc_t, and dh_t = dG_t W_h for the step before
//   weights   dW_g^T = X^T dG and dW_m = dM^T H over all T B rows, with the
//             bias gradients summed in the same pass (k_gemm_tn reads X, dG,
//             dM and H as stored, K outer), the one-hot columns by a
//             deterministic reduction, then the canonical layout
// The forward and per-step products are C[m][n] = sum_k A[m][k] B[n][k] on
// the direct-to-LDS core (both operands K-contiguous: the packing kernel
// also writes W_h^T and W_m^T for them).
// ===========================================================================
namespace {

using GradGemm = GemmD<float, 4, 2, 2, 2, 2>;   // 128 x 64 tiles: the products over all rows
using GradGemmS = GemmD<float, 2, 2, 2, 2, 2>;  // 64 x 64 tiles: the per-step product dG_t . W_h

// out[m][n] = sum_{k < Kpad} A[m][k] B[n][k] for m < M, n < N (Kpad a
// multiple of 32; columns of A and B up to Kpad must be readable, zero
// beyond the data)
// Split K: work-group row y takes columns [y Kpad, (y + 1) Kpad) and writes
// out + y oslice (the caller sums the slices).
template <class C>
__global__ void __launch_bounds__(C::NT) k_gemm_nt(const float* A, long lda, int M, const float* Bm, long ldb,
                                                   int N, int Kpad, float* out, long ldo, long oslice,
                                                   TileMap map) {
  __shared__ __attribute__((aligned(16))) char lds[C::LDS_BYTES];
  int nt, mt;
  if (!tile_of(map, nt, mt)) return;
  A += (long)blockIdx.y * Kpad;
  Bm += (long)blockIdx.y * Kpad;
  out += (long)blockIdx.y * oslice;
  const int n0 = nt * C::BN, m0 = mt * C::BM;
  const SrcX<float> w(Bm, ldb, Kpad, n0, C::BN, N);
  const SrcX<float> x(A, lda, Kpad, m0, C::BM, M);
  f32x4 acc[C::NBW][C::MBW];
  C::run(acc, w, x, Kpad, reinterpret_cast<float*>(lds));
  const int lane = threadIdx.x & 63, r16 = lane & 15, g = lane >> 4;
  const int wn = C::wn(), wmi = C::wm();
#pragma unroll
  for (int j = 0; j < C::MBW; ++j) {
    const int m = m0 + (wmi * C::MBW + j) * 16 + r16;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < C::NBW; ++i) {
      const int n = n0 + (wn * C::NBW + i) * 16 + 4 * g;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (n + v < N) out[(long)m * ldo + n + v] = acc[i][j][v];
    }
  }
}

// N = sum_b min(max(len_b, 0), T) (all B T without lengths)
__global__ void k_len_sum(const int32_t* lengths, int B, int T, float* nout) {
  __shared__ long part[256];
  long s = 0;
  for (int b = threadIdx.x; b < B; b += 256) s += lengths ? min(max(lengths[b], 0), T) : T;
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    long t = 0;
    for (int i = 0; i < 256; ++i) t += part[i];
    nout[0] = (float)t;
  }
}

__device__ __forceinline__ float sig_(float x) { return 1.0f / (1.0f + expf(-x)); }

// forward scan of one (row b, unit u): pre-activations G (packed gate
// order, row r = t B + b, column 4u + q) plus bias and the action's column
// -> activations i, f, tanh g, o in place; c_t into Cs [T+1, B, H]
__global__ void __launch_bounds__(256) k_grad_fwd_scan(float* G, const float* bg, const float* WaT,
                                                       const int32_t* actions, float* Cs, int B, int T, int H,
                                                       int A) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)B * H) return;
  const int b = (int)(idx / H), u = (int)(idx % H);
  const float4 bias = reinterpret_cast<const float4*>(bg)[u];
  float c = 0.f;
  Cs[(long)b * H + u] = 0.f;
  for (int t = 0; t < T; ++t) {
    const long r = (long)t * B + b;
    float4 g = reinterpret_cast<float4*>(G + r * 4 * H)[u];
    const int a = actions[r];
    float4 w = make_float4(0.f, 0.f, 0.f, 0.f);
    if (a >= 0 && a < A) w = reinterpret_cast<const float4*>(WaT + (long)a * 4 * H)[u];
    const float i = sig_(g.x + bias.x + w.x), f = sig_(g.y + bias.y + w.y);
    const float gg = tanhf(g.z + bias.z + w.z), o = sig_(g.w + bias.w + w.w);
    c = f * c + i * gg;
    reinterpret_cast<float4*>(G + r * 4 * H)[u] = make_float4(i, f, gg, o);
    Cs[((long)(t + 1) * B + b) * H + u] = c;
  }
}

// d loss / d head output of one row r = t B + b: for each latent dim j the
// mixture features of packed rows 16 Q J + 16 q + 4 g + v (j = 4J + g,
// feature 4q + v); thread j = Z takes the reward/done block and the padding
// columns.  M holds the head's GEMM outputs and is overwritten with dM.
// lrow [T B, Z+1] receives each (row, dim)'s share of the loss: -loglik_j /
// (N Z), and (se + bce) / N in column Z (0 on padded steps).
template <int KC>
__global__ void __launch_bounds__(256) k_grad_heads(float* M, long ldm, const float* bm, const float* z,
                                                    const float* rewards, const uint8_t* dones,
                                                    const int32_t* lengths, const float* nsum, int B, int T,
                                                    int Z, int Nm, int NmP, float* lrow) {
  constexpr int K = KC, Q = (3 * K + 3) / 4;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)T * B * (Z + 1)) return;
  const long r = idx / (Z + 1);
  const int j = (int)(idx % (Z + 1));
  const int t = (int)(r / B), b = (int)(r % B);
  const float N = nsum[0];
  const bool valid = t < (lengths ? min(max(lengths[b], 0), T) : T) && N > 0.f;
  float* row = M + r * ldm;
  if (j == Z) {
    const int hr = Nm - 16;
    const float rr = row[hr] + bm[hr], rd = row[hr + 1] + bm[hr + 1];
    const float dr = rr - rewards[r], dd = (float)dones[r];
    // softplus(rd) - d rd, stable for either sign of rd
    const float bce = fmaxf(rd, 0.f) + log1pf(expf(-fabsf(rd))) - dd * rd;
    lrow[r * (Z + 1) + Z] = valid ? (dr * dr + bce) / N : 0.f;
    row[hr] = valid ? 2.0f * dr / N : 0.f;
    row[hr + 1] = valid ? (sig_(rd) - dd) / N : 0.f;
    for (int c = hr + 2; c < Nm; ++c) row[c] = 0.f;
    for (int c = Nm; c < NmP; ++c) row[c] = 0.f;
    return;
  }
  const int J = j >> 2, g = j & 3;
  float f[4 * Q];
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int c = 16 * Q * J + 16 * q + 4 * g + v;
      f[4 * q + v] = row[c] + bm[c];
    }
  const float x = z[(long)(t + 1) * B * Z + (long)b * Z + j];  // target z_{t+1, j}
  float mx = -INFINITY;
#pragma unroll
  for (int k = 0; k < K; ++k) mx = fmaxf(mx, f[k]);
  float se = 0.f;
#pragma unroll
  for (int k = 0; k < K; ++k) se += expf(f[k] - mx);
  const float lse_pi = mx + logf(se);
  float joint[K], uu[K], sg[K];
  float jm = -INFINITY;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const float mu = f[K + k], ls = f[2 * K + k];
    sg[k] = expf(ls);
    uu[k] = (x - mu) / sg[k];
    joint[k] = (f[k] - lse_pi) - 0.5f * uu[k] * uu[k] - ls - kHalfLn2Pi;
    jm = fmaxf(jm, joint[k]);
  }
  float sj = 0.f;
#pragma unroll
  for (int k = 0; k < K; ++k) sj += expf(joint[k] - jm);
  const float ll = jm + logf(sj);
  const float s = valid ? -1.0f / (N * (float)Z) : 0.f;  // d loss / d loglik_j
  lrow[r * (Z + 1) + j] = s * ll;
  float d[4 * Q];
#pragma unroll
  for (int k = 0; k < 4 * Q; ++k) d[k] = 0.f;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const float gam = expf(joint[k] - ll), pi = expf(f[k] - lse_pi);
    d[k] = s * (gam - pi);
    d[K + k] = s * gam * uu[k] / sg[k];
    d[2 * K + k] = s * gam * (uu[k] * uu[k] - 1.0f);
  }
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int v = 0; v < 4; ++v) row[16 * Q * J + 16 * q + 4 * g + v] = d[4 * q + v];
}

// LSTM backward of step t for (row b, unit u): with dh = d loss / d h_{t+1}
// (heads + the later steps) and dc = d loss / d c_{t+1} from the later steps,
// writes dG_t (pre-activation gradients, packed gate order) and the new dc
// (dhr: S slices [S, B, H] of the later step's dG . W_h, summed in order)
__global__ void __launch_bounds__(256) k_grad_lstm_back(const float* G, const float* Cs, const float* dhh,
                                                        const float* dhr, int S, float* dc, float* dG, int B,
                                                        int H, int t, int last) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)B * H) return;
  const int b = (int)(idx / H), u = (int)(idx % H);
  const long r = (long)t * B + b;
  const float4 a = reinterpret_cast<const float4*>(G + r * 4 * H)[u];  // i, f, g, o
  const float c1 = Cs[((long)(t + 1) * B + b) * H + u], c0 = Cs[((long)t * B + b) * H + u];
  float dh = dhh[r * H + u];
  if (!last) {
    float sum = 0.f;
    for (int k = 0; k < S; ++k) sum += dhr[(long)k * B * H + (long)b * H + u];
    dh += sum;
  }
  const float dcn = last ? 0.f : dc[(long)b * H + u];
  const float th = tanhf(c1);
  const float d_o = dh * th;
  const float dcc = dcn + dh * a.w * (1.0f - th * th);
  const float d_i = dcc * a.z, d_f = dcc * c0, d_g = dcc * a.x;
  dc[(long)b * H + u] = dcc * a.y;
  reinterpret_cast<float4*>(dG + r * 4 * H)[u] =
      make_float4(d_i * a.x * (1.0f - a.x), d_f * a.y * (1.0f - a.y), d_g * (1.0f - a.z * a.z),
                  d_o * a.w * (1.0f - a.w));
}

// one-hot columns: dWa[a][j] = sum over rows r with action a of dG[r][j].
// Block (256-column tile, row chunk, group of 64 actions): each thread owns
// one column and accumulates the chunk's rows in row order into an LDS slot
// per action; partial [chunk][a][j], summed over the chunks in order.
constexpr int kActGroup = 64;
__global__ void __launch_bounds__(256) k_grad_actions(const float* dG, const int32_t* actions, long R, int H4,
                                                      int A, int nchunk, float* part) {
  __shared__ float acc[kActGroup][256];
  __shared__ int acts[256];
  const int j = blockIdx.x * 256 + threadIdx.x, ch = blockIdx.y, a0 = blockIdx.z * kActGroup;
  const long r0 = R * ch / nchunk, r1 = R * (ch + 1) / nchunk;
  for (int a = 0; a < kActGroup; ++a) acc[a][threadIdx.x] = 0.f;
  for (long rb = r0; rb < r1; rb += 256) {
    __syncthreads();
    const long r = rb + threadIdx.x;
    const int av = r < r1 ? actions[r] : -1;
    acts[threadIdx.x] = (av >= a0 && av < A && av < a0 + kActGroup) ? av - a0 : -1;
    __syncthreads();
    const int n = (int)min((long)256, r1 - rb);
    for (int k = 0; k < n; k += 4) {
      int a[4];
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[q] = (k + q < n && j < H4) ? acts[k + q] : -1;
        v[q] = a[q] >= 0 ? dG[(rb + k + q) * H4 + j] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (a[q] >= 0) acc[a[q]][threadIdx.x] += v[q];
    }
  }
  if (j >= H4) return;
  const int na = min(kActGroup, A - a0);
  for (int a = 0; a < na; ++a) part[((long)ch * A + a0 + a) * H4 + j] = acc[a][threadIdx.x];
}
__global__ void __launch_bounds__(256) k_grad_actions_sum(const float* part, long n, int nchunk, float* out) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int ch = 0; ch < nchunk; ++ch) s += part[(long)ch * n + i];
  out[i] = s;
}

// Fixed-order sum of n floats: block b sums its contiguous piece (each
// thread a strided share, then a tree over the block) into part[b]; one
// block then sums part[0 .. nb) the same way.
constexpr int kFlatBlocks = 512;
__global__ void __launch_bounds__(256) k_flat_sum(const float* x, long n, float* part) {
  __shared__ float red[256];
  const long per = (n + gridDim.x - 1) / gridDim.x;
  const long i0 = (long)blockIdx.x * per, i1 = min(n, i0 + per);
  float acc = 0.f;
  for (long i = i0 + threadIdx.x; i < i1; i += 256) acc += x[i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[blockIdx.x] = red[0];
}

// packed-order gradients -> canonical layout
struct UnpackArgs {
  int Z, H, A, K, Q, Nm, ldk;
  const float *dWgT, *dWa, *dbg, *dWm, *dbm;  // [ldk, 4H], [A, 4H], [4H], [NmP, H], [NmP]
  float *W_g, *b_g, *W_m, *b_m, *w_r, *b_r, *w_d, *b_d;
};
__global__ void __launch_bounds__(256) k_grad_unpack(const UnpackArgs p) {
  const int Z = p.Z, H = p.H, A = p.A, K = p.K, Q = p.Q;
  const long ng = (long)4 * H * (Z + A + H), nm = (long)3 * Z * K * H;
  const long total = ng + 4 * H + nm + 3 * Z * K + 2 * H + 2;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
    long e = i;
    if (e < ng) {  // W_g: canonical row q H + u <- packed row 4u + q
      const int cr = (int)(e / (Z + A + H)), c = (int)(e % (Z + A + H));
      const int pr = 4 * (cr % H) + cr / H;
      float v;
      if (c < Z) v = p.dWgT[(long)c * 4 * H + pr];
      else if (c < Z + A) v = p.dWa[(long)(c - Z) * 4 * H + pr];
      else v = p.dWgT[(long)(Z + c - Z - A) * 4 * H + pr];
      p.W_g[e] = v;
      continue;
    }
    e -= ng;
    if (e < 4 * H) {
      p.b_g[e] = p.dbg[4 * (e % H) + e / H];
      continue;
    }
    e -= 4 * H;
    auto prow = [&](long cr) {  // canonical mixture row p ZK + j K + k -> packed row
      const int pp = (int)(cr / ((long)Z * K)), rem = (int)(cr % ((long)Z * K));
      const int j = rem / K, k = rem % K, f = pp * K + k;
      return 16 * Q * (j >> 2) + 16 * (f >> 2) + 4 * (j & 3) + (f & 3);
    };
    if (e < nm) {
      const long cr = e / H;
      p.W_m[e] = p.dWm[(long)prow(cr) * H + e % H];
      continue;
    }
    e -= nm;
    if (e < 3 * Z * K) {
      p.b_m[e] = p.dbm[prow(e)];
      continue;
    }
    e -= 3 * Z * K;
    if (e < H) { p.w_r[e] = p.dWm[(long)(p.Nm - 16) * H + e]; continue; }
    e -= H;
    if (e < H) { p.w_d[e] = p.dWm[(long)(p.Nm - 15) * H + e]; continue; }
    e -= H;
    if (e == 0) p.b_r[0] = p.dbm[p.Nm - 16];
    else p.b_d[0] = p.dbm[p.Nm - 15];
  }
}

// K slices of an M x N x Kpad product: doubled (up to kGradMaxSplit) while
// the tiles number under 512 and the 32-column chunks divide evenly
constexpr int kGradMaxSplit = 8;
template <class C = GradGemm>
int split_of(int M, int N, int Kpad, long target = 512) {
  const long tiles = (long)((N + C::BN - 1) / C::BN) * ((M + C::BM - 1) / C::BM);
  const int chunks = Kpad / 32;
  int S = 1;
  while (S < kGradMaxSplit && tiles * S < target && chunks % (2 * S) == 0 && chunks / (2 * S) >= 4) S *= 2;
  return S;
}

// the per-step product: its tile shape and K slices
using BpttGemm = GradGemmS;
int bptt_split(int B, int H) { return split_of<BpttGemm>(B, H, 4 * H, 256); }

// out (ldo) = A . B^T in S K-slices; S > 1 writes slice y to out + y oslice
template <class C = GradGemm>
hipError_t gemm_nt_slices(const char* name, const float* A, long lda, int M, const float* Bm, long ldb, int N,
                          int Kpad, int S, float* out, long ldo, long oslice, hipStream_t s) {
  const int Ks = Kpad / S;
  const TileMap map = tile_map((N + C::BN - 1) / C::BN, (M + C::BM - 1) / C::BM, (size_t)N * Ks * 4);
  return launch(name, k_gemm_nt<C>, dim3(grid_of(map), (unsigned)S), dim3(C::NT), 0, s, A, lda, M, Bm, ldb, N,
                Ks, out, ldo, oslice, map);
}

// x[0 .. n) = 0
__global__ void __launch_bounds__(256) k_zero(float* x, long n) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) x[i] = 0.f;
}

// ===========================================================================
// k_gemm_tn: out[m][n] = sum over rows k of A[k][m] B[k][n], both operands
// row-major with the reduction over their rows (the weight-gradient products
// over the T B rows read their activation and gradient matrices as stored,
// no transposed copies).  K slice s covers rows [s Ks, (s+1) Ks) and writes
// its own partial [M, N] (summed in fp64 afterwards).  128 x 64 tiles, four
// waves of 64 x 32; chunks of 16 rows reach LDS by LDS-DMA in a ring of four
// stages.  A fragment read takes rows 4g + j, j < 4, of a chunk (one MFMA
// each): the 16-byte pieces of staged row k are XOR-permuted by ((k/4) mod 4)
// * 4, so that the four lane groups g read four distinct 64-byte bank
// windows.  SUMA / SUMB: the work-groups of the first tile column / row also
// sum A's / B's columns over their rows (an extra MFMA block against ones)
// into colsum partials [S, M] / [S, N].  Work-group -> tile: XCD x takes
// the slices s = x mod 8, each slice's tiles m fastest, so that a slice's
// rows are shared in one L2.
// ===========================================================================
constexpr int kTnBM = 128, kTnBN = 64, kTnBK = 16, kTnStages = 4;
constexpr int kTnStageBytes = (kTnBM + kTnBN) * kTnBK * 4;  // 12 KB: A rows, then B rows

struct TnArgs {
  const float* A;
  const float* Bm;
  long lda, ldb, K;
  int Ks, S, M, N, ntm, ntn;
  float* part;  // [S, M, N] partials (ldp = N)
  float* csA;   // [S, M] or null
  float* csB;   // [S, N] or null
};

__global__ void __launch_bounds__(256) k_gemm_tn(const TnArgs p) {
  __shared__ __attribute__((aligned(1024))) char lds[kTnStages * kTnStageBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, r16 = lane & 15;
  const int x = blockIdx.x & 7, r = blockIdx.x >> 3;
  const int per = p.ntm * p.ntn;
  const int sl = x + 8 * (r / per);
  if (sl >= p.S) return;
  const int nt = (r % per) / p.ntm, mt = (r % per) % p.ntm;
  const int m0 = mt * kTnBM, n0 = nt * kTnBN;
  const long k0 = (long)sl * p.Ks;
  const long k1 = min(p.K, k0 + (long)p.Ks);
  const int nk = (int)((k1 - k0 + kTnBK - 1) / kTnBK);
  // the slice's rows only: rows past k1 (and the tail of the last row) read zero
  const u32x4 ra = rsrc_words(p.A + k0 * p.lda, (uint32_t)((k1 - k0) * p.lda * 4));
  const u32x4 rb = rsrc_words(p.Bm + k0 * p.ldb, (uint32_t)((k1 - k0) * p.ldb * 4));
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) char*)lds);
  // this wave's three DMA instructions per chunk: q < 8 stage A rows 2q, 2q+1
  // (32 pieces each), q >= 8 B rows 4(q-8) .. +3 (16 pieces each)
  bool isa[3];
  uint32_t off[3];
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    const int q = wave * 3 + t;
    isa[t] = q < 8;
    if (isa[t]) {
      const int row = 2 * q + (lane >> 5), pc = (lane & 31) ^ (((row >> 2) & 3) << 2);
      off[t] = (uint32_t)(row * p.lda + m0) * 4u + 16u * (uint32_t)pc;
    } else {
      const int row = 4 * (q - 8) + (lane >> 4), pc = (lane & 15) ^ (((row >> 2) & 3) << 2);
      off[t] = (uint32_t)(row * p.ldb + n0) * 4u + 16u * (uint32_t)pc;
    }
  }
  const uint32_t stepa = (uint32_t)(kTnBK * p.lda) * 4u, stepb = (uint32_t)(kTnBK * p.ldb) * 4u;
  auto issue = [&](int kc) {
    const uint32_t base = lds0 + (uint32_t)(kc % kTnStages) * kTnStageBytes + (uint32_t)wave * 3u * 1024u;
#pragma unroll
    for (int t = 0; t < 3; ++t)
      dma16(isa[t] ? ra : rb, off[t] + (uint32_t)kc * (isa[t] ? stepa : stepb), base + 1024u * t);
  };
#pragma unroll
  for (int c = 0; c < kTnStages - 1; ++c)
    if (c < nk) issue(c);

  const int wm = wave >> 1, wn = wave & 1;
  const bool suma = p.csA && nt == 0 && wn == 0;  // wave-uniform
  const bool sumb = p.csB && mt == 0 && wm == 0;
  f32x4 acc[4][2], cs[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc[i][0] = acc[i][1] = cs[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // lane byte offsets inside a stage: A element (4g + j, (wm 4 + i) 16 + r16),
  // B element (4g + j, (wn 2 + jb) 16 + r16)
  uint32_t oa[4], ob[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) oa[i] = (uint32_t)(4 * g * 512 + (((wm * 4 + i) ^ g) & 7) * 64 + r16 * 4);
#pragma unroll
  for (int jb = 0; jb < 2; ++jb) ob[jb] = (uint32_t)(kTnBM * kTnBK * 4 + 4 * g * 256 + (((wn * 2 + jb) ^ g) & 3) * 64 + r16 * 4);
  for (int kc = 0; kc < nk; ++kc) {
    const int young = min(kTnStages - 2, nk - 1 - kc);
    if (young >= 2) vm_wait<6>();
    else if (young == 1) vm_wait<3>();
    else vm_wait<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" : : : "memory");
    if (kc + kTnStages - 1 < nk) issue(kc + kTnStages - 1);
    const char* buf = lds + (kc % kTnStages) * kTnStageBytes;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float a[4], b[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const float*>(buf + oa[i] + j * 512);
#pragma unroll
      for (int jb = 0; jb < 2; ++jb) b[jb] = *reinterpret_cast<const float*>(buf + ob[jb] + j * 256);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) acc[i][jb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[jb], acc[i][jb], 0, 0, 0);
      if (suma) {
#pragma unroll
        for (int i = 0; i < 4; ++i) cs[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], 1.0f, cs[i], 0, 0, 0);
      }
      if (sumb) {
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) cs[jb] = __builtin_amdgcn_mfma_f32_16x16x4f32(1.0f, b[jb], cs[jb], 0, 0, 0);
      }
    }
  }
  // lane (g, r16) holds C[4g + v][r16]: rows m, columns n
  float* part = p.part + (long)sl * p.M * p.N;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      const int n = n0 + (wn * 2 + jb) * 16 + r16;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + (wm * 4 + i) * 16 + 4 * g + v;
        if (m < p.M && n < p.N) part[(long)m * p.N + n] = acc[i][jb][v];
      }
    }
  if (suma && r16 == 0) {  // every column of C holds A's column sums
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + (wm * 4 + i) * 16 + 4 * g + v;
        if (m < p.M) p.csA[(long)sl * p.M + m] = cs[i][v];
      }
  }
  if (sumb && g == 0) {  // every row of C holds B's column sums
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      const int n = n0 + (wn * 2 + jb) * 16 + r16;
      if (n < p.N) p.csB[(long)sl * p.N + n] = cs[jb][0];
    }
  }
}

// The weight-gradient products reduce over all T B rows.  A K slice
// accumulates its products in fp32, one MFMA after another, so its rounding
// error grows with the slice's length; the slices are therefore kept to at
// most kMaxSliceK rows and summed in fp64 (relative error of the product
// then ~ 1e-5 of the terms' magnitude at T B = 65536).
constexpr int kMaxSliceK = 2048;
int split_long(int M, int N, int Kpad) {
  int S = split_of(M, N, Kpad);
  while (Kpad / S > kMaxSliceK && (Kpad / 32) % (2 * S) == 0) S *= 2;
  return S;
}

// out[m][n] = sum_s part[s][m][n] in slice order, accumulated in fp64
__global__ void __launch_bounds__(256) k_sum_slices(const float* part, int S, int M, int N, float* out, long ldo) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)M * N) return;
  const long mn = (long)M * N;
  double acc = 0.0;
  for (int k = 0; k < S; ++k) acc += (double)part[k * mn + i];
  out[(i / N) * ldo + i % N] = (float)acc;
}

// out (ldo) = A . B^T, split over K through `part` ([S, M, N]) when that
// fills the chip better, or (long_k) to bound the fp32 accumulation chains
hipError_t gemm_nt(const float* A, long lda, int M, const float* Bm, long ldb, int N, int Kpad, float* out,
                   long ldo, float* part, hipStream_t s, bool long_k = false) {
  const int S = part ? (long_k ? split_long(M, N, Kpad) : split_of(M, N, Kpad)) : 1;
  if (S == 1) return gemm_nt_slices("grad_gemm", A, lda, M, Bm, ldb, N, Kpad, 1, out, ldo, 0, s);
  const hipError_t e = gemm_nt_slices("grad_gemm", A, lda, M, Bm, ldb, N, Kpad, S, part, N, (long)M * N, s);
  if (e != hipSuccess) return e;
  return launch("grad_sum", k_sum_slices, dim3((unsigned)(((long)M * N + 255) / 256)), dim3(256), 0, s, part, S, M,
                N, out, ldo);
}

// K slices of a product over K rows (kMaxSliceK rows each)
inline int tn_slices(long K) { return (int)((K + kMaxSliceK - 1) / kMaxSliceK); }

// out (ldo) = A^T B over the K rows of both (A [K, lda] with M used columns,
// B [K, ldb] with N), through the slice partials `part` ([S, M, N]) summed in
// fp64; with csA (csB) also the column sums of A (B) into colsum ([M] or [N],
// slice partials in cpart [S, M or N]).
hipError_t gemm_tn(const float* A, long lda, int M, const float* Bm, long ldb, int N, long K, float* part,
                   float* out, long ldo, bool sum_a, bool sum_b, float* cpart, float* colsum, hipStream_t s) {
  if (sum_a && sum_b) return hipErrorInvalidValue;  // one colsum register set per wave
  TnArgs a{};
  a.A = A; a.Bm = Bm; a.lda = lda; a.ldb = ldb; a.K = K;
  a.Ks = kMaxSliceK;
  a.S = tn_slices(K);
  a.M = M; a.N = N;
  a.ntm = (M + kTnBM - 1) / kTnBM;
  a.ntn = (N + kTnBN - 1) / kTnBN;
  a.part = part;
  a.csA = sum_a ? cpart : nullptr;
  a.csB = sum_b ? cpart : nullptr;
  const long nwg = (long)((a.S + 7) / 8) * 8 * a.ntm * a.ntn;
  hipError_t e = launch("grad_gemm_tn", k_gemm_tn, dim3((unsigned)nwg), dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  e = launch("grad_sum", k_sum_slices, dim3((unsigned)(((long)M * N + 255) / 256)), dim3(256), 0, s,
             (const float*)part, a.S, M, N, out, ldo);
  if (e != hipSuccess || !(sum_a || sum_b)) return e;
  const int nc = sum_a ? M : N;
  return launch("grad_sum", k_sum_slices, dim3((unsigned)((nc + 255) / 256)), dim3(256), 0, s, (const float*)cpart,
                a.S, 1, nc, colsum, (long)nc);
}

template <int KC>
hipError_t launch_heads_k(float* M, long ldm, const float* bm, const float* z, const float* rewards,
                          const uint8_t* dones, const int32_t* lengths, const float* nsum, int B, int T, int Z,
                          int Nm, int NmP, float* lrow, hipStream_t s) {
  const long n = (long)T * B * (Z + 1);
  return launch("grad_heads", k_grad_heads<KC>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, M, ldm,
                bm, z, rewards, dones, lengths, nsum, B, T, Z, Nm, NmP, lrow);
}

}  // namespace

// row chunks of the one-hot column reduction: about 512 work-groups
static int act_chunks(const Layout& L) {
  const int tiles = (4 * L.H + 255) / 256 * ((L.A + kActGroup - 1) / kActGroup);
  return std::min(64, std::max(1, 512 / tiles));
}

size_t grad_workspace(const Layout& L, int B, int T, char* ws, GradWs* G) {
  const long TB = (long)T * B, TBp = (TB + 31) / 32 * 32;
  const int H = L.H, H4 = 4 * H, NmP = (L.Nm + 31) / 32 * 32;
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = wm_align256(o + bytes); return at; };
  const size_t oG = take((size_t)TB * H4 * 4), oC = take((size_t)(T + 1) * B * H * 4);
  const size_t oM = take((size_t)TB * NmP * 4), odG = take((size_t)TB * H4 * 4);
  const size_t odhh = take((size_t)TB * H * 4), odh = take((size_t)B * H * 4), odc = take((size_t)B * H * 4);
  const size_t odWgT = take((size_t)L.ldk * H4 * 4), odWa = take((size_t)L.A * H4 * 4);
  const size_t odWm = take((size_t)NmP * H * 4), odbg = take((size_t)H4 * 4), odbm = take((size_t)NmP * 4);
  const size_t opart = take((size_t)std::max(kFlatBlocks, tn_slices(TB)) * std::max(H4, NmP) * 4);
  const size_t oapart = take((size_t)act_chunks(L) * L.A * H4 * 4);
  // split-K partials: the largest of the products that split, and the
  // per-step slices of dG_t . W_h (always)
  auto split_need = [](int M, int N, int Kpad, bool long_k = false) {
    const int S = long_k ? split_long(M, N, Kpad) : split_of(M, N, Kpad);
    return S > 1 ? (size_t)S * M * N : (size_t)0;
  };
  const size_t nsplit = std::max({(size_t)bptt_split(B, H) * B * H, split_need((int)TB, H4, L.ldk),
                                  split_need((int)TB, L.Nm, L.ldh), split_need((int)TB, H, NmP),
                                  (size_t)tn_slices(TB) * L.ldk * H4, (size_t)tn_slices(TB) * NmP * H});
  const size_t osplit = take(nsplit * 4);
  const size_t on = take(16);
  const size_t ofwd = take((size_t)TB * (L.Z + 1) * 4);  // loss terms [TB, Z+1]
  if (ws && G) {
    auto f = [&](size_t at) { return reinterpret_cast<float*>(ws + at); };
    G->G = f(oG); G->Cs = f(oC); G->M = f(oM); G->dG = f(odG); G->dhh = f(odhh); G->dh = f(odh);
    G->dc = f(odc);
    G->dWgT = f(odWgT); G->dWa = f(odWa); G->dWm = f(odWm); G->dbg = f(odbg); G->dbm = f(odbm);
    G->part = f(opart); G->apart = f(oapart); G->split = f(osplit); G->nsum = f(on); G->fwd = f(ofwd);
  }
  return o;
}

hipError_t launch_nll_grad(const Packed& P, NllBufs N, const GradWs& G, const GradOut& out, hipStream_t s) {
  const Layout& L = P.L;
  const int B = N.B, T = N.T, Z = L.Z, H = L.H, A = L.A, H4 = 4 * H;
  const long TB = (long)T * B, TBp = (TB + 31) / 32 * 32;
  const int NmP = (L.Nm + 31) / 32 * 32;
  const char* base = reinterpret_cast<const char*>(P.base);
  const float* Wg = reinterpret_cast<const float*>(base + L.off_Wg);
  const float* WaT = reinterpret_cast<const float*>(base + L.off_WaT);
  const float* bg = reinterpret_cast<const float*>(base + L.off_bg);
  const float* Wm = reinterpret_cast<const float*>(base + L.off_Wm);
  const float* bm = reinterpret_cast<const float*>(base + L.off_bm);
  const float* WhT = reinterpret_cast<const float*>(base + L.off_WhT);  // [H, 4H]
  const float* WmT = reinterpret_cast<const float*>(base + L.off_WmT);  // [H, NmP]
  const float* X = reinterpret_cast<const float*>(N.x);
  const float* Hn = X + (long)B * L.ldx + Z;  // h_1 .. h_T: rows of X_1 .. X_T from column Z
  hipError_t e;
#define WM_TRY(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  // forward recurrence: X (z_t | h_t) for every step. Where the persistent
  // kernel serves it, it also leaves the gate activations and c_{t+1} of
  // every step; otherwise they are recomputed from X (pre-activations of
  // every step in one GEMM, then a scan that applies the gates and records
  // c_t).
  const bool traced = persist_usable(L, B, true);
  N.g_trace = traced ? G.G : nullptr;
  N.c_trace = traced ? G.Cs : nullptr;
  WM_TRY(nll_impl<float>(P, N, s, false));
  WM_TRY(launch("grad_len", k_len_sum, dim3(1), dim3(256), 0, s, N.lengths, B, T, G.nsum));
  if (traced) {
    WM_TRY(launch("grad_zero", k_zero, dim3((unsigned)(((long)B * H + 255) / 256)), dim3(256), 0, s, G.Cs,
                  (long)B * H));  // c_0
  } else {
    WM_TRY(gemm_nt(X, L.ldx, (int)TB, Wg, L.ldk, H4, L.ldk, G.G, H4, G.split, s));
    WM_TRY(launch("grad_scan", k_grad_fwd_scan, dim3((unsigned)(((long)B * H + 255) / 256)), dim3(256), 0, s,
                  G.G, bg, WaT, N.actions, G.Cs, B, T, H, A));
  }
  // head outputs of every h_{t+1}, then d loss / d output in place
  WM_TRY(gemm_nt(Hn, L.ldx, (int)TB, Wm, L.ldh, L.Nm, L.ldh, G.M, NmP, G.split, s));
  switch (L.K) {
#define WM_HK(k)                                                                                       \
  case k:                                                                                              \
    WM_TRY(launch_heads_k<k>(G.M, NmP, bm, N.z, N.rewards, N.dones, N.lengths, G.nsum, B, T, Z, L.Nm, \
                             NmP, G.fwd, s));                                                          \
    break;
    WM_HK(1) WM_HK(2) WM_HK(3) WM_HK(4) WM_HK(5) WM_HK(6) WM_HK(7) WM_HK(8)
#undef WM_HK
    default: return hipErrorInvalidValue;
  }
  if (out.loss) {  // the loss: a fixed-order sum of its (row, dim) terms
    WM_TRY(launch("grad_loss", k_flat_sum, dim3(kFlatBlocks), dim3(256), 0, s, (const float*)G.fwd,
                  TB * (Z + 1), G.part));
    WM_TRY(launch("grad_loss", k_flat_sum, dim3(1), dim3(256), 0, s, (const float*)G.part, (long)kFlatBlocks,
                  out.loss));
  }
  // d loss / d h_{t+1} through the heads: dM [TB, NmP] . W_m (the packed
  // W_m^T [H, NmP], zero columns past Nm)
  WM_TRY(gemm_nt(G.M, NmP, (int)TB, WmT, NmP, H, NmP, G.dhh, H, G.split, s));
  // back through time (the packed W_h^T [H, 4H])
  const unsigned eg = (unsigned)(((long)B * H + 255) / 256);
  const int Sb = bptt_split(B, H);  // K slices of dG_t . W_h, summed by the next step's kernel
  for (int t = T - 1; t >= 0; --t) {
    WM_TRY(launch("grad_lstm", k_grad_lstm_back, dim3(eg), dim3(256), 0, s, G.G, G.Cs, G.dhh, G.split, Sb, G.dc,
                  G.dG, B, H, t, t == T - 1 ? 1 : 0));
    if (t > 0)
      WM_TRY(gemm_nt_slices<BpttGemm>("grad_gemm_bptt", G.dG + (long)t * B * H4, H4, B, WhT, H4, H, H4, Sb, G.split, H,
                            (long)B * H, s));
  }
  // dW_g^T [ldk, 4H] = X^T . dG over all rows, read as stored; the bias
  // gradient (dG's column sums) from the same pass
  WM_TRY(gemm_tn(X, L.ldx, L.ldk, G.dG, H4, H4, TB, G.split, G.dWgT, H4, false, true, G.part, G.dbg, s));
  const int nch = act_chunks(L);
  WM_TRY(launch("grad_actions", k_grad_actions,
                dim3((unsigned)((H4 + 255) / 256), (unsigned)nch, (unsigned)((A + kActGroup - 1) / kActGroup)),
                dim3(256), 0, s, G.dG, N.actions, TB, H4, A, nch, G.apart));
  WM_TRY(launch("grad_actions", k_grad_actions_sum, dim3((unsigned)(((long)A * H4 + 255) / 256)), dim3(256), 0,
                s, G.apart, (long)A * H4, nch, G.dWa));
  // dW_m [NmP, H] = dM^T . H over all rows, and the head bias gradient
  // (dM's column sums)
  WM_TRY(gemm_tn(G.M, NmP, NmP, Hn, L.ldx, H, TB, G.split, G.dWm, H, true, false, G.part, G.dbm, s));
  // canonical layout
  const UnpackArgs u{Z, H, A, L.K, L.Q, L.Nm, L.ldk, G.dWgT, G.dWa, G.dbg, G.dWm, G.dbm,
                     out.W_g, out.b_g, out.W_m, out.b_m, out.w_r, out.b_r, out.w_d, out.b_d};
  WM_TRY(launch("grad_unpack", k_grad_unpack, dim3(1024), dim3(256), 0, s, u));
#undef WM_TRY
  return hipSuccess;
}

}  // namespace wm
