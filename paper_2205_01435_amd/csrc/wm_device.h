// Device helpers for the World-Model dream kernels (gfx950 / CDNA4).
//
// MFMA fragments: both GEMM operands are K-contiguous ([rows, K] row-major),
// and every lane feeds 16 bytes per operand per step:
//   fp32  v_mfma_f32_16x16x4_f32, four issues per 16-wide K slice; lane group
//         g = lane / 16 owns k = 4g .. 4g+3 of the slice (one per issue);
//   bf16  v_mfma_f32_16x16x32_bf16, one issue per 32-wide K slice; lane group
//         g owns k = 8g .. 8g+7.
// Any fixed assignment of k to (lane group, slot) gives the same dot product
// as long as both operands use it, which they do.
// Output block (16 x 16, fp32): lane l holds rows 4*(l/16) + v, v = 0..3, of
// column l % 16.  Rows index output features (weights are the A operand) and
// columns index batch rows, so each lane holds 4 consecutive features of one
// batch row; the packed weight layouts put what an epilogue needs together
// into those quartets.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wm {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint16_t bf16_t;  // storage type of bfloat16 values

// ---------------------------------------------------------------------------
// bfloat16 storage: round to nearest, ties to even; NaN stays NaN.  gfx950
// converts in hardware (v_cvt_pk_bf16_f32, two values per instruction).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}
// (bits of a) | (bits of b) << 16
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
  bf16x2 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }
__device__ __forceinline__ float round_bf16(float f) { return bf16_bits_to_f32(f32_to_bf16_bits(f)); }

__device__ __forceinline__ uint4 pack8_bf16(float4 a, float4 b) {
  uint4 r;
  r.x = pack2_bf16(a.x, a.y);
  r.y = pack2_bf16(a.z, a.w);
  r.z = pack2_bf16(b.x, b.y);
  r.w = pack2_bf16(b.z, b.w);
  return r;
}

template <typename DT> struct DType;
template <> struct DType<float> {
  static constexpr int VEC = 4;  // elements per 16 bytes
  __device__ static float load(const float* p, long i) { return p[i]; }
  __device__ static float round(float x) { return x; }
  __device__ static void store(float* p, long i, float x) { p[i] = x; }
};
template <> struct DType<bf16_t> {
  static constexpr int VEC = 8;
  __device__ static float load(const bf16_t* p, long i) { return bf16_bits_to_f32(p[i]); }
  __device__ static float round(float x) { return round_bf16(x); }
  __device__ static void store(bf16_t* p, long i, float x) { p[i] = (bf16_t)f32_to_bf16_bits(x); }
};

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64 multiplies, high halves crossed with the other words and the key,
// key bumped by the Weyl constants between rounds.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c.x, hi0 = __umulhi(0xD2511F53u, c.x);
    const uint32_t lo1 = 0xCD9E8D57u * c.z, hi1 = __umulhi(0xCD9E8D57u, c.z);
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
  }
  return c;
}

struct Rng {
  uint32_t k0, k1;
  __device__ __forceinline__ uint4 block(uint32_t blk, uint32_t step, uint32_t traj,
                                         uint32_t stream) const {
    return philox4x32_10(make_uint4(blk, step, traj, stream), k0, k1);
  }
};

// ((x >> 9) + 1/2) * 2^-23: midpoint of one of 2^23 cells of (0, 1), exact.
__device__ __forceinline__ float word_to_uniform(uint32_t x) {
  return ((float)(x >> 9) + 0.5f) * 0x1p-23f;
}
__device__ __forceinline__ uint32_t word_of(uint4 w, int i) {
  return i == 0 ? w.x : (i == 1 ? w.y : (i == 2 ? w.z : w.w));
}
// Gumbel score -ln(-ln u) as -ln(ln 2) - ln 2 * log2(-log2 u), on the
// hardware log2 (v_log_f32, accurate to about an ulp in relative terms also
// near 1, where the library logf relies on it too).  The uniforms here are
// normal numbers in [2^-24, 1), so the library's denormal and infinity
// handling is not needed.  Over all 2^23 uniforms of word_to_uniform the
// largest error against float64 is 2.0e-6 absolute, 2.1e-7 relative to
// max(1, |score|) (library logf: 1.9e-6 and 2.9e-7).
__device__ __forceinline__ float gumbel(float u) {
  return fmaf(-0.69314718055994531f, __builtin_amdgcn_logf(-__builtin_amdgcn_logf(u)), 0.36651292058166435f);
}
__device__ __forceinline__ float sigmoidf(float x) { return 1.0f / (1.0f + expf(-x)); }

// Fast LSTM nonlinearities on the hardware base-2 exponential and reciprocal
// (v_exp_f32, v_rcp_f32, about 1 ulp each): relative error below 1e-6 for
// |x| <= 20.  tanh switches to its odd Taylor polynomial for |x| < 1/8,
// where 1 - exp(-2|x|) would cancel (truncation error below 2e-9).
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float fsigmoid(float x) { return frcp(1.0f + fexp(-x)); }
__device__ __forceinline__ float ftanh(float x) {
  const float ax = fabsf(x);
  const float t = fexp(-2.0f * ax);
  const float big = (1.0f - t) * frcp(1.0f + t);
  const float x2 = x * x;
  const float small = ax * (1.0f + x2 * (-1.0f / 3.0f + x2 * (2.0f / 15.0f + x2 * (-17.0f / 315.0f))));
  return copysignf(ax < 0.125f ? small : big, x);
}

// tanh as 1 - 2 / (1 + exp(2x)), without the small-|x| branch: about 2.5e-7
// absolute error (relative accuracy is lost near 0 to the cancellation),
// three VALU and two transcendental instructions against ten and two.  For
// the bf16 cells, whose h is rounded to bf16 (relative step 2^-9) right away.
__device__ __forceinline__ float ftanh_abs(float x) {
  return 1.0f - 2.0f * frcp(1.0f + __builtin_amdgcn_exp2f(x * 2.88539008177792681f));
}
// LSTM cell of the bf16 kernels: c' = sigmoid(f) c + sigmoid(i) tanh(g) and
// h' = sigmoid(o) tanh(c'), each written over one common denominator:
//   c' = (c (1 + Ei)(1 + G) + (1 - G)(1 + Ef)) / ((1 + Ef)(1 + Ei)(1 + G)),
//   h' = (1 - C) / ((1 + Eo)(1 + C)),
// with Ex = exp(-x) for the sigmoids, G = exp(-2g) and C = exp(-2c') for the
// tanhs: five exponentials and two reciprocals instead of five and five.
// Pre-activations and c' are clamped to +-15 first, where the sigmoid and
// tanh are within 3.1e-7 of their limits, so that the products stay finite;
// the result is within about 1e-6 of the separate functions (h is rounded to
// bf16, relative step 2^-9, right after).
constexpr float kCellClamp = 15.0f;
__device__ __forceinline__ void lstm_cell_fused(float pi, float pf, float pg, float po, float c,
                                                float& cn, float& hn) {
  constexpr float L2E = 1.44269504088896341f;
  const float xi = __builtin_amdgcn_fmed3f(pi, -kCellClamp, kCellClamp);
  const float xf = __builtin_amdgcn_fmed3f(pf, -kCellClamp, kCellClamp);
  const float xg = __builtin_amdgcn_fmed3f(pg, -kCellClamp, kCellClamp);
  const float xo = __builtin_amdgcn_fmed3f(po, -kCellClamp, kCellClamp);
  const float ai = 1.0f + __builtin_amdgcn_exp2f(xi * -L2E);
  const float af = 1.0f + __builtin_amdgcn_exp2f(xf * -L2E);
  const float ao = 1.0f + __builtin_amdgcn_exp2f(xo * -L2E);
  const float G = __builtin_amdgcn_exp2f(xg * (-2.0f * L2E));
  const float d1 = ai * (1.0f + G);
  cn = __builtin_fmaf(c, d1, (1.0f - G) * af) * frcp(af * d1);
  const float C = __builtin_amdgcn_exp2f(__builtin_amdgcn_fmed3f(cn, -kCellClamp, kCellClamp) * (-2.0f * L2E));
  hn = (1.0f - C) * frcp(ao * (1.0f + C));
}

// the cell's tanh for activation type DT
template <typename DT>
__device__ __forceinline__ float ftanh_cell(float x) {
  if constexpr (sizeof(DT) == 4) return ftanh(x);
  else return ftanh_abs(x);
}

enum : uint32_t {
  STREAM_CONTROLLER = 0,  // controller Gumbel noise (action, or xfer of the two-level controller)
  STREAM_COMPONENT = 1,
  STREAM_GAUSS = 2,
  STREAM_DONE = 3,
  STREAM_LOCATION = 4     // two-level controller: location Gumbel noise
};

// ---------------------------------------------------------------------------
// MFMA step on one 16-byte fragment per operand.
// ---------------------------------------------------------------------------
template <typename DT> struct Mfma;
template <> struct Mfma<float> {
  static constexpr int KSLICE = 16;
  __device__ __forceinline__ static void step(f32x4& acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  }
};
template <> struct Mfma<bf16_t> {
  static constexpr int KSLICE = 32;
  __device__ __forceinline__ static void step(f32x4& acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
  }
};

// ---------------------------------------------------------------------------
// Buffer (range-checked) loads: a 16-byte load at a byte offset at or beyond
// the resource's size returns zeros without touching memory, which replaces
// per-load bounds branches and 64-bit address arithmetic.  Offsets are 32-bit
// (resources are at most 2^31 bytes); kOffNone addresses nothing.
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOffNone = 0x80000000u;

__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 bload16(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}
__device__ __forceinline__ uint2 bload8(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
}
__device__ __forceinline__ uint32_t bload4(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
}
__device__ __forceinline__ uint32_t bload1(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b8(r, (int)off, 0, 0);
}
__device__ __forceinline__ uint32_t bload2(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
}
// Stores at an offset at or beyond the resource's size are dropped.
__device__ __forceinline__ void bstore4(rsrc_t r, uint32_t off, uint32_t v) {
  __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)off, 0, 0);
}
__device__ __forceinline__ void bstore2(rsrc_t r, uint32_t off, uint32_t v) {
  __builtin_amdgcn_raw_buffer_store_b16((unsigned short)v, r, (int)off, 0, 0);
}
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void bstore8(rsrc_t r, uint32_t off, uint2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{v.x, v.y}, r, (int)off, 0, 0);
}
__device__ __forceinline__ void bstore16(rsrc_t r, uint32_t off, uint4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{v.x, v.y, v.z, v.w}, r, (int)off, 0, 0);
}
__device__ __forceinline__ float4 as_float4(uint4 v) {
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
}
__device__ __forceinline__ uint4 as_uint4(float4 v) {
  return make_uint4(__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w));
}
__device__ __forceinline__ uint4 operator|(uint4 a, uint4 b) {
  return make_uint4(a.x | b.x, a.y | b.y, a.z | b.z, a.w | b.w);
}

// 16 bytes of DT activations from a source of element type S at byte offset
// `off` (fp32 sources are converted to DT: two 16-byte loads when DT is bf16).
template <typename DT, typename S>
__device__ __forceinline__ uint4 bload_x16(rsrc_t r, uint32_t off) {
  if constexpr (sizeof(S) == sizeof(DT)) {
    return bload16(r, off);
  } else {
    const uint4 a = bload16(r, off);
    const uint4 b = bload16(r, off == kOffNone ? kOffNone : off + 16u);
    return pack8_bf16(make_float4(__uint_as_float(a.x), __uint_as_float(a.y), __uint_as_float(a.z),
                                  __uint_as_float(a.w)),
                      make_float4(__uint_as_float(b.x), __uint_as_float(b.y), __uint_as_float(b.z),
                                  __uint_as_float(b.w)));
  }
}

// ---------------------------------------------------------------------------
// GEMM operand sources.  Each addresses the rows of one work-group tile
// through a buffer resource, so that rows past the valid ones and columns at
// or past Kpad read as zero, with straight-line code.  row(i) gives the
// per-row part of the byte offset, load(row, k, Kpad) the 16 bytes of
// columns k .. k+VEC-1 (k a multiple of VEC).
//   SrcX   one row-major DT matrix with a row stride of ld elements (the
//          weights, and the activation matrix [q(z) | h | 0]);
//   SrcZH  float32 z [M, Z] followed by float32 h [M, H], converted to DT
//          (the standalone controller step, whose inputs are two tensors).
// ---------------------------------------------------------------------------
template <typename DT_>
struct SrcX {
  using DT = DT_;
  using Row = uint32_t;
  static constexpr bool kTwo = false;
  rsrc_t r;
  const DT* base;  // first row of the tile
  uint32_t bytes;  // readable bytes from base
  uint32_t ldb;    // row stride in bytes
  // rows m0 .. m0+rows-1 of x, clipped to M; `span` readable columns per row
  __device__ SrcX(const DT* x, long ld, long span, int m0, int rows, int M) {
    const long mval = max(0, min(rows, M - m0));
    ldb = (uint32_t)(ld * (long)sizeof(DT));
    base = x + (long)m0 * ld;
    bytes = mval ? (uint32_t)(((mval - 1) * ld + span) * (long)sizeof(DT)) : 0u;
    r = make_rsrc(base, bytes);
  }
  __device__ Row row(int i) const { return (uint32_t)i * ldb; }
  __device__ uint4 load(Row ro, int k, int Kpad) const {
    return bload16(r, k < Kpad ? ro + (uint32_t)k * (uint32_t)sizeof(DT) : kOffNone);
  }
};

template <typename DT_>
struct SrcZH {
  using DT = DT_;
  using Row = uint2;
  static constexpr bool kTwo = true;
  rsrc_t rz, rh;
  int Z, Kx;
  uint32_t zb, hb;  // row strides in bytes
  __device__ SrcZH(const float* z, const float* h, int Z_, int H, int m0, int rows, int M) {
    const long mval = max(0, min(rows, M - m0));
    Z = Z_;
    Kx = Z_ + H;
    zb = (uint32_t)Z_ * 4u;
    hb = (uint32_t)H * 4u;
    rz = make_rsrc(z + (long)m0 * Z_, (uint32_t)(mval * Z_ * 4));
    rh = make_rsrc(h + (long)m0 * H, (uint32_t)(mval * H * 4));
  }
  __device__ Row row(int i) const { return make_uint2((uint32_t)i * zb, (uint32_t)i * hb); }
  __device__ uint4 load(Row ro, int k, int /*Kpad*/) const {
    const bool inz = k < Z, inh = k >= Z && k < Kx;
    return bload_x16<DT, float>(rz, inz ? ro.x + (uint32_t)k * 4u : kOffNone) |
           bload_x16<DT, float>(rh, inh ? ro.y + (uint32_t)(k - Z) * 4u : kOffNone);
  }
};


// ---------------------------------------------------------------------------
// Mixture sampling of one latent dim j of one trajectory at one step:
// Gumbel-max component pick on pi-logit / tau (stream 1, uniform j*K + k),
// then mu + exp(log sigma) * eps with eps from Box-Muller on the stream-2 pair
// (2p, 2p+1) that contains j (cos for even j, sin for odd j).
// mixture_noise draws the random part (independent of the head GEMM, so it
// can be issued early); mixture_pick finishes from the dim's features
// f = 0 .. 4Q-1 (pi-logits, means, log sigmas, padding), biased.
// ---------------------------------------------------------------------------
struct MdnNoise {
  float g[8];  // Gumbel noise of components 0 .. K-1 (K <= 8)
  float eps;   // standard normal of dim j
};

// Gumbel noise of components 0 .. K-1 of dim j, one Philox block per four
// consecutive uniforms of the dim.
__device__ __forceinline__ void component_noise(MdnNoise& n, const Rng& rng, int K, uint32_t step,
                                                uint32_t traj, int j) {
  uint32_t cur = 0xffffffffu;
  uint4 w = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    n.g[k] = 0.f;
    if (k < K) {
      const uint32_t idx = (uint32_t)j * K + k;
      if ((idx >> 2) != cur) {
        cur = idx >> 2;
        w = rng.block(cur, step, traj, STREAM_COMPONENT);
      }
      n.g[k] = gumbel(word_to_uniform(word_of(w, idx & 3)));
    }
  }
}

// Box-Muller on one stream-2 word pair: (cos deviate, sin deviate), which
// belong to the pair's even and odd dim.
__device__ __forceinline__ float2 box_muller(uint32_t w1, uint32_t w2) {
  const float u1 = word_to_uniform(w1);
  const float u2 = word_to_uniform(w2);
  const float r = sqrtf(-2.0f * logf(u1));
  float sn, cs;
  sincospif(2.0f * u2, &sn, &cs);
  return make_float2(r * cs, r * sn);
}

// The standard normals of the four dims 4J .. 4J+3 (one stream-2 block).
__device__ __forceinline__ float4 gauss_group(const Rng& rng, uint32_t step, uint32_t traj, int J) {
  const uint4 wg = rng.block((uint32_t)J, step, traj, STREAM_GAUSS);
  const float2 e01 = box_muller(wg.x, wg.y), e23 = box_muller(wg.z, wg.w);
  return make_float4(e01.x, e01.y, e23.x, e23.y);
}

__device__ __forceinline__ MdnNoise mixture_noise(const Rng& rng, int K, uint32_t step, uint32_t traj,
                                                  int j) {
  MdnNoise n;
  component_noise(n, rng, K, step, traj, j);
  const uint4 wg = rng.block((uint32_t)j >> 2, step, traj, STREAM_GAUSS);
  const float2 e = box_muller(word_of(wg, j & 2), word_of(wg, (j & 2) + 1));
  n.eps = (j & 1) ? e.y : e.x;
  return n;
}

// sig scales the normal deviate (1 = plain mixture; sqrt(tau) for the
// sigma temperature)
template <int Q>
__device__ __forceinline__ float mixture_pick(int K, float tau, const MdnNoise& n,
                                              const float (&feat)[4 * Q], float sig = 1.0f) {
  float best = -INFINITY;
  int kbest = 0;
  if (tau == 1.0f) {  // x / 1 == x: the same scores without the divisions
#pragma unroll
    for (int f = 0; f < 4 * Q && f < 8; ++f) {
      if (f < K) {
        const float sc = feat[f] + n.g[f];
        if (sc > best) { best = sc; kbest = f; }
      }
    }
  } else {
#pragma unroll
    for (int f = 0; f < 4 * Q && f < 8; ++f) {
      if (f < K) {
        const float sc = feat[f] / tau + n.g[f];
        if (sc > best) { best = sc; kbest = f; }
      }
    }
  }
  float mu = 0.f, ls = 0.f;
#pragma unroll
  for (int f = 0; f < 4 * Q; ++f) {
    if (f == K + kbest) mu = feat[f];
    if (f == 2 * K + kbest) ls = feat[f];
  }
  return mu + expf(ls) * (n.eps * sig);
}

// ---------------------------------------------------------------------------
// LDS-DMA: buffer loads that write straight into LDS (no staging registers,
// no LDS store instructions).
// ---------------------------------------------------------------------------
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// Buffer resource words for inline assembly (same fields as make_rsrc).
__device__ __forceinline__ u32x4 rsrc_words(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  u32x4 r;
  r.x = (uint32_t)a;
  r.y = (uint32_t)(a >> 32) & 0xffffu;
  r.z = bytes;
  r.w = 0x00020000u;
  return r;
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane from the buffer at byte offset voff into LDS at
// lds + 16 * lane (lds is wave-uniform).  Out-of-range offsets load zeros.
// Issued as inline assembly so that the compiler does not wait for these
// loads before every LDS read; callers wait with vm_wait<N>() instead.
__device__ __forceinline__ void dma16(u32x4 rs, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rs)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// vm_wait with a run-time bound (clamped to 0 .. 63).
__device__ __forceinline__ void vm_wait_n(int n) {
  switch (n <= 0 ? 0 : (n >= 63 ? 63 : n)) {
#define WM_VMW(k) case k: vm_wait<k>(); break;
    WM_VMW(0) WM_VMW(1) WM_VMW(2) WM_VMW(3) WM_VMW(4) WM_VMW(5) WM_VMW(6) WM_VMW(7)
    WM_VMW(8) WM_VMW(9) WM_VMW(10) WM_VMW(11) WM_VMW(12) WM_VMW(13) WM_VMW(14) WM_VMW(15)
    WM_VMW(16) WM_VMW(17) WM_VMW(18) WM_VMW(19) WM_VMW(20) WM_VMW(21) WM_VMW(22) WM_VMW(23)
    WM_VMW(24) WM_VMW(25) WM_VMW(26) WM_VMW(27) WM_VMW(28) WM_VMW(29) WM_VMW(30) WM_VMW(31)
    WM_VMW(32) WM_VMW(33) WM_VMW(34) WM_VMW(35) WM_VMW(36) WM_VMW(37) WM_VMW(38) WM_VMW(39)
    WM_VMW(40) WM_VMW(41) WM_VMW(42) WM_VMW(43) WM_VMW(44) WM_VMW(45) WM_VMW(46) WM_VMW(47)
    WM_VMW(48) WM_VMW(49) WM_VMW(50) WM_VMW(51) WM_VMW(52) WM_VMW(53) WM_VMW(54) WM_VMW(55)
    WM_VMW(56) WM_VMW(57) WM_VMW(58) WM_VMW(59) WM_VMW(60) WM_VMW(61) WM_VMW(62) WM_VMW(63)
#undef WM_VMW
  }
}

}  // namespace wm
