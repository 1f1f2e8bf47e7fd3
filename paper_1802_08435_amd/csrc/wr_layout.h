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
// Head workgroups (NH): head j evaluates the gates of every unit (redundantly,
// identically in all heads), owns rows [j*HR, j*HR+HR) of O1 and O3, the
// matching columns of O2 and O4, and coarse rows [j*GR, j*GR+GR) of R's
// fine-input half (R_c[:, fine], needed right after y_f is known).  Rows of R
// are indexed per half: coarse row cr = g*Hh + i <-> R row g*H + i, fine row
// fr = g*Hh + i <-> R row g*H + Hh + i (g = u, r, e).
// Unit workgroups (NU): unit workgroup k owns coarse rows [k*UR, +UR) of R's
// coarse-input half (GA rows) and fine rows [k*UR, +UR) of all of R (GF rows).
//
// Matrices are stored bf16 as MFMA fragments (v_mfma_f32_16x16x32_bf16 with
// the matrix as operand B): fragment (mt, kt) covers rows 16*mt .. 16*mt+15 and
// input columns 32*kt .. 32*kt+31; lane l holds row 16*mt + l%16, columns
// 32*kt + 8*(l/16) .. +7 (16 bytes).  A fragment is 1 KiB, lanes in order.
// ---------------------------------------------------------------------------
#define WR_THREADS 512    // 8 waves per workgroup
#define WR_HR 32          // O1 / O3 rows per head workgroup (2 row tiles)
#define WR_GR 96          // R_c[:, fine] rows per head workgroup (6 row tiles)
#define WR_UR 32          // GA rows and GF rows per unit workgroup (2 row tiles)
#define WR_XALIGN 64      // exchange regions aligned to 64 words (512 B)
#define WR_MAXNH 16       // partial-logit sets summed per draw
#define WR_FRAG 1024      // bytes per MFMA fragment

struct PersistPlan {
  int H, Hh, KT;          // KT = Hh / 32 column tiles per input half
  int NH, NU;
  // head LDS block (bytes): O1 slice, O3 slice, R_c fine-half slice
  int hb_o1, hb_o3, hb_rcf, h_bytes;
  // unit LDS block (bytes): GA rows (coarse half), GF rows (both halves)
  int ub_ga, ub_gf, u_bytes;
  // exchange words
  int x_yc, x_yf, x_ga, x_gf, x_gcf, x_aec, x_aef, x_pc, x_pf, x_words;
  // LDS bytes
  int lds_h, lds_u, lds;
};

WR_HD inline int wr_rup(int x, int m) { return (x + m - 1) / m * m; }

WR_HD inline bool persist_plan(int H, PersistPlan* P) {
  if (H <= 0 || H % 128) return false;
  P->H = H;
  P->Hh = H / 2;
  P->KT = P->Hh / 32;
  if (P->Hh % WR_HR || (3 * P->Hh) % WR_UR) return false;
  P->NH = P->Hh / WR_HR;
  P->NU = 3 * P->Hh / WR_UR;
  if (P->NH > WR_MAXNH || P->Hh > WR_THREADS) return false;
  P->hb_o1 = 0;
  P->hb_o3 = P->hb_o1 + (WR_HR / 16) * P->KT * WR_FRAG;
  P->hb_rcf = P->hb_o3 + (WR_HR / 16) * P->KT * WR_FRAG;
  P->h_bytes = P->hb_rcf + (WR_GR / 16) * P->KT * WR_FRAG;
  P->ub_ga = 0;
  P->ub_gf = (WR_UR / 16) * P->KT * WR_FRAG;
  P->u_bytes = P->ub_gf + (WR_UR / 16) * 2 * P->KT * WR_FRAG;
  int o = 0;
  auto take = [&](int n) { int r = o; o += wr_rup(n, WR_XALIGN); return r; };
  P->x_yc = take(P->Hh);
  P->x_yf = take(P->Hh);
  P->x_ga = take(3 * P->Hh);
  P->x_gf = take(3 * P->Hh);
  P->x_gcf = take(3 * P->Hh);
  P->x_aec = take(P->Hh);
  P->x_aef = take(P->Hh);
  P->x_pc = take(P->NH * 256);
  P->x_pf = take(P->NH * 256);
  P->x_words = o;
  // head: weights, h[H], z[256], zh[256], op[8][32], rp[4][96], ov[32], bs[64], misc[16]
  P->lds_h = P->h_bytes + 4 * (H + 256 + 256 + 8 * WR_HR + 4 * WR_GR + WR_HR + 64 + 16);
  // unit: weights, y[H], partials[2][8][32], misc[16]
  P->lds_u = P->u_bytes + 4 * (H + 2 * 8 * WR_UR + 16);
  P->lds = P->lds_h > P->lds_u ? P->lds_h : P->lds_u;
  return P->lds <= 160 * 1024;
}
