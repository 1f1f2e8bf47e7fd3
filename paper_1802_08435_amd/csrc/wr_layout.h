// Memory layouts shared by the host packer and the kernels of libwavernn.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define WR_HD __host__ __device__
#else
#define WR_HD
#endif

// ---------------------------------------------------------------------------
// Single-workgroup kernel: one fp32 image copied to LDS, then scratch arrays.
// Offsets in floats, each region 16-byte aligned.
// ---------------------------------------------------------------------------
struct SmallLayout {
  int H;
  int Rt, I, bias, O1t, O2t, O3t, O4t, b1, b2, b3, b4, image_floats;  // image (weights)
  int add, G, h, hn, hid, z, w, C, total_floats;                       // scratch
};

WR_HD inline int wr_take(int& o, int n) {
  int r = o;
  o += (n + 3) & ~3;
  return r;
}

WR_HD inline SmallLayout small_layout(int H) {
  SmallLayout L;
  L.H = H;
  const int Hh = H / 2;
  int o = 0;
  L.Rt = wr_take(o, 3 * H * H);   // Rt[j][row] = R[row][j], rows g*H + i
  L.I = wr_take(o, 9 * H);        // I[row][3], masked
  L.bias = wr_take(o, 3 * H);
  L.O1t = wr_take(o, Hh * Hh);    // O1t[j][k] = O1[k][j]
  L.O2t = wr_take(o, Hh * 256);   // O2t[j][v] = O2[v][j]
  L.O3t = wr_take(o, Hh * Hh);
  L.O4t = wr_take(o, Hh * 256);
  L.b1 = wr_take(o, Hh);
  L.b2 = wr_take(o, 256);
  L.b3 = wr_take(o, Hh);
  L.b4 = wr_take(o, 256);
  L.image_floats = o;
  L.add = wr_take(o, 3 * H);
  L.G = wr_take(o, 3 * H);
  L.h = wr_take(o, H);
  L.hn = wr_take(o, H);
  L.hid = wr_take(o, Hh);
  L.z = wr_take(o, 256);
  L.w = wr_take(o, 256);
  L.C = wr_take(o, 256);
  L.total_floats = o;
  return L;
}

// ---------------------------------------------------------------------------
// Persistent multi-workgroup kernel.
//
// Roles: NU unit workgroups (U), NC coarse-head workgroups (HC), NF fine-head
// workgroups (HF).  U workgroup k owns units [k*UC, k*UC+UC) of the coarse half
// and the same offsets of the fine half, i.e. 6*UC rows of R (3 gates x 2
// halves).  Local row lr = g*2*UC + half*UC + j  <->  R row g*H + half*H/2 + k*UC + j.
// HC workgroup j owns rows [j*HC, j*HC+HC) of O1 and the matching columns of
// O2 (a split of O2's inner dimension); HF likewise for O3 / O4.
//
// Dense matrices are stored bf16 in "row-block" order: 8 rows x 8 lanes per
// block, lane l = 8*r + q covers columns q*SEG .. q*SEG+SEG-1 of one half of
// the input (SEG = K/8), in chunks of 8 bf16 (16 bytes):
//   chunk(rb, i, l) at ((rb * CPL + i) * 64 + l) * 16 bytes,  CPL = SEG / 8.
// A wave reading chunk i of a block touches 64 consecutive 16-byte slots.
// ---------------------------------------------------------------------------
#define WR_UC 8           // units per half per U workgroup
#define WR_THREADS 384    // 6 waves: one row-block of 8 rows per wave in U
#define WR_XALIGN 64      // exchange regions aligned to 64 words (512 B)

struct PersistPlan {
  int H, Hh, SEG, CPL;    // SEG = Hh / 8 columns per lane, CPL = SEG / 8 chunks
  int NU, NC, NF;         // workgroups per role
  int HCR, HCP;           // head rows per HC/HF workgroup, padded to 8
  int u_rows;             // 6 * WR_UC
  int u_half_bytes;       // one half (coarse or fine columns) of a U block
  int u_bytes;            // U weight block bytes
  int h1_bytes;           // head first-layer block bytes (HCP rows x Hh)
  int h2_bytes;           // head second-layer block bytes (256 x HCP)
  int h_bytes;            // h1 + h2
  // exchange words
  int x_yc, x_yf, x_pc, x_pf, x_words;
  // LDS bytes
  int lds_u, lds_h, lds;
};

WR_HD inline int wr_rup(int x, int m) { return (x + m - 1) / m * m; }

WR_HD inline bool persist_plan(int H, PersistPlan* P) {
  if (H <= 0 || H % 128) return false;
  P->H = H;
  P->Hh = H / 2;
  P->SEG = P->Hh / 8;
  P->CPL = P->SEG / 8;
  if (P->Hh % WR_UC) return false;
  P->NU = P->Hh / WR_UC;
  // head split: at most 32 rows per head workgroup
  int nc = 1;
  while (P->Hh / nc > 32 || P->Hh % nc) ++nc;
  if (nc > 16) return false;   // partial-logit sets read per draw
  P->NC = P->NF = nc;
  P->HCR = P->Hh / nc;
  P->HCP = wr_rup(P->HCR, 8);
  P->u_rows = 6 * WR_UC;
  P->u_half_bytes = P->u_rows * P->Hh * 2;
  P->u_bytes = 2 * P->u_half_bytes;
  P->h1_bytes = P->HCP * P->Hh * 2;
  P->h2_bytes = 256 * P->HCP * 2;
  P->h_bytes = P->h1_bytes + P->h2_bytes;
  P->x_yc = 0;
  P->x_yf = wr_rup(P->Hh, WR_XALIGN);
  P->x_pc = 2 * P->x_yf;
  P->x_pf = P->x_pc + P->NC * 256;
  P->x_words = P->x_pf + P->NF * 256;
  // U: weights, h[H], Gc[3UC], Gf[2][3UC], add[6UC], I[6UC][3], z[256], misc
  P->lds_u = P->u_bytes + 4 * (H + 3 * WR_UC + 6 * WR_UC + 6 * WR_UC + 18 * WR_UC + 256 + 64);
  // H: weights, y[Hh], o[HCP], b[HCP], misc
  P->lds_h = P->h_bytes + 4 * (P->Hh + 2 * P->HCP + 64);
  P->lds = P->lds_u > P->lds_h ? P->lds_u : P->lds_h;
  return P->lds <= 160 * 1024;
}
