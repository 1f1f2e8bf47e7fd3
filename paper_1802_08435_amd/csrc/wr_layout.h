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
// Head workgroups (NH = Hh / 64): every head evaluates the gates of every unit
// (redundantly and identically), so all heads hold the whole hidden state
// without exchanging it.  Head j owns rows [64j, 64j+64) of O1 and O3 and the
// matching 64 columns of O2 and O4, kept in VGPRs as MFMA fragments; it
// publishes 256 partial logits per half, and every head sums the NH partials
// in the same order and draws the same class.
// Unit workgroups (NU): R is cut into 16-row tiles, each tile within one gate
// and one half (coarse rows: R row g*H + i, i < Hh; fine rows: g*H + Hh + i).
// Unit k owns coarse tiles [k*UCT, +UCT) and fine tiles [k*UCT, +UCT) over all
// H columns, so it publishes finished pre-activations R h (+ bias and
// conditioning for the u and r gates) of those rows for the next step.
//
// Matrices are stored bf16 as MFMA fragments (v_mfma_f32_16x16x32_bf16 with
// the matrix as operand B): fragment (mt, kt) covers rows 16*mt .. 16*mt+15 and
// input columns 32*kt .. 32*kt+31; lane l holds row 16*mt + l%16, columns
// 32*kt + 8*(l/16) .. +7 (16 bytes).  A fragment is 1 KiB, lanes in order.
// ---------------------------------------------------------------------------
#define WR_THREADS 512    // 8 waves per workgroup
#define WR_HROWS 64       // O1 / O3 rows per head workgroup (4 row tiles)
#define WR_XALIGN 64      // exchange regions aligned to 64 words (512 B)
#define WR_FRAG 1024      // bytes per MFMA fragment
#define WR_MAXUCT 3       // coarse (and fine) row tiles per unit workgroup (waves 3, 7 stay free)

struct PersistPlan {
  int H, Hh, KT, KH;      // KT = Hh / 32 column tiles per half, KH = KT / 2
  int NH, NU, UCT, NCT;   // heads, units, row tiles per unit and half, row tiles per half (3 Hh / 16)
  int grid;               // workgroups launched: head j at block 8j, units on the others
  int hw_frags;           // head fragments per wave: O1[KH], O3[KH], O2[4], O4[4]
  int u_lds_w;            // unit LDS weight block: coarse tiles x coarse columns, fine tiles x all columns
  int x_yc, x_yf, x_ga, x_gf, x_pc, x_pf, x_words;   // exchange regions (64-bit words)
  int x_ps;               // words between the partial-logit blocks of consecutive heads
  int lds_h, lds_u, lds;  // LDS bytes
};

WR_HD inline int wr_rup(int x, int m) { return (x + m - 1) / m * m; }

// Block index of head j and the role of block b (head index, or unit index + NH, or -1 idle).
WR_HD inline int wr_role(const PersistPlan& P, int b) {
  if (b % 8 == 0 && b / 8 < P.NH) return b / 8;
  int before = (b + 7) / 8;                 // head blocks with index < b
  if (before > P.NH) before = P.NH;
  int k = b - before;
  return k < P.NU ? P.NH + k : -1;
}

WR_HD inline bool persist_plan(int H, PersistPlan* P) {
  if (H <= 0 || H % 128) return false;
  P->H = H;
  P->Hh = H / 2;
  P->KT = P->Hh / 32;
  P->KH = P->KT / 2;
  P->NH = P->Hh / WR_HROWS;
  P->NCT = 3 * P->Hh / 16;
  if (P->NH > 16 || P->Hh > WR_THREADS - 64) return false;   // the last wave draws, free of gate work
  P->hw_frags = 2 * P->KH + 8;
  // head LDS: y_c and y_f operand images (KT fragments each), relu image (2),
  // first-layer partials [2][64], logit sums [2][256], logits [256],
  // y [448], misc [16], uniforms [2][64][2], targets [2][64]
  P->lds_h = (2 * P->KT + 2) * WR_FRAG + 4 * (2 * 64 + 3 * 256 + 448 + 16 + 256 + 128);
  P->UCT = 0;
  for (int u = WR_MAXUCT; u >= 1; --u) {
    if (P->NCT % u) continue;
    int w = 3 * u * P->KT * WR_FRAG;
    int l = w + 2 * P->KT * WR_FRAG + 4 * 16;
    if (l <= 160 * 1024) { P->UCT = u; P->u_lds_w = w; P->lds_u = l; break; }
  }
  if (!P->UCT) return false;
  P->NU = P->NCT / P->UCT;
  int g = 8 * (P->NH - 1) + 1;
  while (g - P->NH < P->NU) ++g;
  P->grid = g;
  int o = 0;
  auto take = [&](int n) { int r = o; o += wr_rup(n, WR_XALIGN); return r; };
  P->x_yc = take(P->Hh);
  P->x_yf = take(P->Hh);
  P->x_ga = take(3 * P->Hh);
  P->x_gf = take(3 * P->Hh);
  P->x_ps = 256;
  P->x_pc = take(P->NH * P->x_ps);
  P->x_pf = take(P->NH * P->x_ps);
  P->x_words = o;
  P->lds = P->lds_h > P->lds_u ? P->lds_h : P->lds_u;
  return P->lds <= 160 * 1024;
}
