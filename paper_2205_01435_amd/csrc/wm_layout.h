// Packed (kernel-side) weight layout of libwm, shared by the packing and the
// compute kernels.  All matrices are row-major with K contiguous, padded with
// zero columns to a multiple of 64 elements so that every K tile is whole.
//
//   Wg  [4H, ldk]  gate rows interleaved per hidden unit: packed row 4u + q
//                  is canonical row q*H + u (q = i, f, g, o), so the four
//                  gates of one unit land in one lane's output quartet;
//                  columns z | h (the one-hot block is moved to WaT).
//   WaT [A, 4H]    the one-hot block transposed (same interleave): adding
//                  row a is the product with onehot(a).
//   bg  [4H]       fp32, interleaved like Wg.
//   Wm  [Nm, ldh]  mixture head.  Latent dims are taken in groups of four;
//                  group J owns 16*Q rows and row 16*Q*J + 16*q + 4*g + v
//                  holds feature f = 4*q + v of dim 4*J + g, where features
//                  0..K-1 are pi-logits, K..2K-1 means, 2K..3K-1 log sigmas
//                  and the rest zero (Q = ceil(3K / 4)).  One MFMA output
//                  quartet per lane then carries one dim's features.  A final
//                  16-row block holds w_r (row 0) and w_d (row 1).
//   bm  [Nm]       fp32, same row order (b_r, b_d in the final block).
//   Wc  [Nc, ldk]  controller rows 0..Ac-1 (columns z | h), row Ac = [0 | w_r],
//                  row Ac+1 = [0 | w_d], zero rows up to Nc = roundup(Ac+2, 16).
//                  Ac = A, or N + 1 + L for the two-level controller (N+1
//                  xfer rows, the last the NO-OP, then L location rows; the
//                  world model's actions are then the A = N L pairs).
//   bc  [Nc]       fp32: b_c (Ac), b_r, b_d, zeros.
//   fp32 only, for the training gradient's products against transposed
//   weights (written by the same packing pass):
//   WhT [H, 4H]    Wg's h columns transposed: WhT[i][r] = Wg[r][Z + i].
//   WmT [H, NmP]   Wm transposed, NmP = roundup(Nm, 32) (zero columns past
//                  Nm): WmT[i][r] = Wm[r][i].
//
// Activations live in one matrix per step, X [rows, ldx] in the same element
// type: columns 0..Z-1 hold q(z), Z..Z+H-1 hold h, the rest zero, so that the
// gate and controller GEMMs read X from column 0 (K = ldk <= ldx) and the
// mixture head reads it from column Z (K = ldh <= ldx - Z).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace wm {

struct Layout {
  int Z, H, A, K, dt;  // dt: 0 fp32, 1 bf16
  int esz;             // bytes per matrix element
  int Kx;              // Z + H
  int ldk;             // roundup(Kx, 64)
  int ldh;             // roundup(H, 64)
  int ldx;             // roundup(Z + ldh, 64): row stride of the activation matrix
  int Q;               // ceil(3K / 4)
  int Nm;              // 16 Q (Z / 4) + 16
  int N, Lc;           // two-level controller: xfers and locations (N = 0: one level)
  int Ac;              // controller logit rows: A, or N + 1 + Lc
  int Nc;              // roundup(Ac + 2, 16)
  int NmP;             // roundup(Nm, 32)
  size_t off_Wg, off_WaT, off_bg, off_Wm, off_bm, off_Wc, off_bc;
  size_t off_WhT, off_WmT;  // fp32 layouts only (else equal to total)
  size_t total;
};

static inline size_t wm_align256(size_t x) { return (x + 255) & ~(size_t)255; }
static inline int wm_roundup(int x, int m) { return (x + m - 1) / m * m; }

static inline Layout make_layout(int Z, int H, int A, int K, int dt, int N = 0, int Lc = 0) {
  Layout L;
  L.Z = Z; L.H = H; L.A = A; L.K = K; L.dt = dt;
  L.N = N; L.Lc = Lc;
  L.Ac = N > 0 ? N + 1 + Lc : A;
  L.esz = dt == 0 ? 4 : 2;
  L.Kx = Z + H;
  L.ldk = wm_roundup(L.Kx, 64);
  L.ldh = wm_roundup(H, 64);
  L.ldx = wm_roundup(Z + L.ldh, 64);
  L.Q = (3 * K + 3) / 4;
  L.Nm = 16 * L.Q * (Z / 4) + 16;
  L.Nc = wm_roundup(L.Ac + 2, 16);
  size_t o = 0;
  L.off_Wg = o;  o = wm_align256(o + (size_t)4 * H * L.ldk * L.esz);
  L.off_WaT = o; o = wm_align256(o + (size_t)A * 4 * H * L.esz);
  L.off_bg = o;  o = wm_align256(o + (size_t)4 * H * 4);
  L.off_Wm = o;  o = wm_align256(o + (size_t)L.Nm * L.ldh * L.esz);
  L.off_bm = o;  o = wm_align256(o + (size_t)L.Nm * 4);
  L.off_Wc = o;  o = wm_align256(o + (size_t)L.Nc * L.ldk * L.esz);
  L.off_bc = o;  o = wm_align256(o + (size_t)L.Nc * 4);
  L.NmP = wm_roundup(L.Nm, 32);
  L.off_WhT = o;
  if (dt == 0) o = wm_align256(o + (size_t)H * 4 * H * 4);
  L.off_WmT = o;
  if (dt == 0) o = wm_align256(o + (size_t)H * L.NmP * 4);
  L.total = o;
  return L;
}

}  // namespace wm
