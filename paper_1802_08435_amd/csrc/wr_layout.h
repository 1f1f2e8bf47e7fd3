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
// Mirror workgroups (NM, the dense batch-1 plan only; 0 in the fused and
// block-sparse plans): mirror j draws c_t from the heads' partial logits as
// every head does, evaluates the gates of the fine half itself and forms the
// coarse rows' products with y_f, R[g*H + i][Hh + c] y_f[c] for i < Hh, of 12
// coarse row tiles (192 rows: mirror j owns coarse row tiles 12j .. 12j + 11),
// which it publishes straight to the heads.  The units then publish only the
// coarse columns' part of the coarse rows (as soon as y_c is in) and the
// whole fine rows, so y_f no longer has to reach the units and come back
// before the next step's coarse gates.  Wave w of a mirror holds row tiles
// 12j + 3(w % 4) .. +2 over the fine column tiles of half w / 4 (KT / 2 each).
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
#define WR_MTILES 12      // coarse row tiles per mirror workgroup (3 Hh / 16 = 12 NH of them)

struct PersistPlan {
  int H, Hh, KT, KH;      // KT = Hh / 32 column tiles per half, KH = column tiles per head wave
  int RT, HR, KO, GU;     // head: row tiles (HR = 16 RT rows of O1 / O3), O2 / O4 column tiles
                          // (HR / 32), gate units per gate thread
  int NH, NU, UCT, NCT;   // heads, units, row tiles per unit and half, row tiles per half (3 Hh / 16)
  int NM, mw_frags;       // mirrors (0: none) and their fragments per wave (3 row tiles x KT / 2)
  int NK;                 // slices of O1 / O3 rows (Hh / HR): the partial logits per half
  int SR, SL, NRC, NRF;   // block-sparse units: rows per unit, lanes per row, block slots per lane
                          // (coarse columns, fine columns); 0 for the dense kernel
  int BH, BW, BR, u_wb;   // block-sparse units: block shape (4 x 4 or 16 x 1), block-rows per unit,
                          // bytes of the weights before the block-column indices
  int grid;               // workgroups launched: head j at block 8j + hx, units on the others
  int hx, uxm;            // placement: heads on XCD hx, units on the XCDs of the bits of uxm
  int hw_frags;           // head fragments per wave: O1[KH], O3[KH], O2[2 KO], O4[2 KO]
  int u_lds_w;            // unit LDS block: dense R tiles, or the block-sparse records
  int x_yc, x_yf, x_ga, x_gf, x_pc, x_pf, x_words;   // exchange regions (32-bit words)
  int x_hf;               // with mirrors: the coarse rows' products with y_f [3 Hh]
  int x_xcc;              // the XCD of each head and mirror, published at the start
  int x_ps;               // words between the partial-logit blocks of consecutive heads
  int x_gfs, x_pfs;       // with mirrors the fine rows' words and the fine partial logits are
                          // double-buffered by step parity: words between the two buffers (0: one)
  int lds_h, lds_u, lds_m, lds;  // LDS bytes
};

// Double-buffered words of step s (the fine rows' pre-activations and the fine
// partial logits when mirrors read them too): buffer s mod 2, tagged with the
// parity of the buffer's generation s / 2 + 1.  A writer of step s + 2 has
// waited, through its own inputs, for every reader of step s (see the head
// and mirror roles), and the generation bit tells step s from step s - 2.
WR_HD inline int wr_dbuf(int64_t s, int stride) { return (int)(s & 1) * stride; }
WR_HD inline uint32_t wr_dtag(int64_t s, int stride) {
  return stride ? (uint32_t)(s >> 1) + 1u : (uint32_t)s + 1u;
}

WR_HD inline int wr_rup(int x, int m) { return (x + m - 1) / m * m; }

// Block index of head j and the role of block b (head index, mirror index +
// NH, unit index + NH + NM, or -1 idle).
// Placement.  Blocks are dealt round-robin over the 8 XCDs (block b runs on
// XCD b % 8), so lead block i (head i < NH, then mirror i - NH) sits at block
// 8 i + hx, and bit x of uxm admits units on the other blocks of XCD x.  Unit
// blocks below b:
WR_HD inline int wr_units_below(const PersistPlan& P, int b) {
  const int NL = P.NH + P.NM;
  int n = (b / 8) * __builtin_popcount(P.uxm & 255) + __builtin_popcount(P.uxm & ((1 << (b % 8)) - 1));
  if (P.uxm >> P.hx & 1) {
    const int leads = (b + 7 - P.hx) / 8;   // blocks b' < b with b' % 8 == hx
    n -= leads < NL ? leads : NL;
  }
  return n;
}
// The role of block b: head index, mirror index + NH, unit index + NH + NM, or
// -1 (idle: returns at once).
WR_HD inline int wr_role(const PersistPlan& P, int b) {
  const int NL = P.NH + P.NM;
  if (b % 8 == P.hx && b / 8 < NL) return b / 8;
  if (!(P.uxm >> (b % 8) & 1)) return -1;
  const int k = wr_units_below(P, b);
  return k < P.NU ? NL + k : -1;
}
// Set a placement and the smallest grid that holds every head, mirror and unit.
WR_HD inline void wr_place(PersistPlan* P, int hx, int uxm) {
  P->hx = hx;
  P->uxm = uxm;
  int g = 8 * (P->NH + P->NM - 1) + hx + 1;
  while (wr_units_below(*P, g) < P->NU) ++g;
  P->grid = g;
}

WR_HD inline bool persist_plan(int H, PersistPlan* P) {
  if (H <= 0 || H % 128) return false;
  P->H = H;
  P->Hh = H / 2;
  P->KT = P->Hh / 32;
  P->KH = P->KT / 2;
  P->NH = P->Hh / WR_HROWS;
  P->NK = P->NH;
  P->RT = 4;
  P->HR = WR_HROWS;
  P->KO = 2;
  P->GU = 1;
  P->SR = P->SL = P->NRC = P->NRF = 0;
  P->BH = P->BW = P->BR = P->u_wb = 0;
  P->NCT = 3 * P->Hh / 16;
  if (P->NH > 16 || P->Hh > WR_THREADS - 64) return false;   // the last wave draws, free of gate work
  P->NM = P->NCT / WR_MTILES;                                 // = NH
  P->mw_frags = 3 * (P->KT / 2);
  P->hw_frags = 2 * P->KH + 8;
  // head LDS: y_c and y_f operand images (KT fragments each), relu image (2),
  // first-layer partials [2][64], logit sums [2][256], logits [256],
  // y [448], misc [16], uniforms [2][64][2], targets [2][64]
  P->lds_h = (2 * P->KT + 2) * WR_FRAG + 4 * (2 * 64 + 3 * 256 + 448 + 16 + 256 + 128);
  P->UCT = 0;
  for (int u = WR_MAXUCT; u >= 1; --u) {
    if (P->NCT % u) continue;
    int w = 2 * u * P->KT * WR_FRAG;
    int l = w + 2 * P->KT * WR_FRAG + 4 * 16;
    if (l <= 160 * 1024) { P->UCT = u; P->u_lds_w = w; P->lds_u = l; break; }
  }
  if (!P->UCT) return false;
  P->NU = P->NCT / P->UCT;
  // mirror LDS: y_f operand image (KT fragments), products of the two column
  // halves [2][192], logits [256], misc [16], uniforms [2][64][2], targets [2][64]
  P->lds_m = P->KT * WR_FRAG + 4 * (2 * 16 * WR_MTILES + 256 + 16 + 256 + 128);
  wr_place(P, 0, 255);
  int o = 0;
  auto take = [&](int n) { int r = o; o += wr_rup(n, WR_XALIGN); return r; };
  P->x_yc = take(P->Hh);
  P->x_yf = take(P->Hh);
  P->x_ga = take(3 * P->Hh);
  P->x_gfs = wr_rup(3 * P->Hh, WR_XALIGN);
  P->x_gf = take(2 * P->x_gfs);
  P->x_hf = take(3 * P->Hh);
  P->x_xcc = take(P->NH + P->NM);
  P->x_ps = 256;
  P->x_pc = take(P->NH * P->x_ps);
  P->x_pfs = P->NH * P->x_ps;
  P->x_pf = take(2 * P->x_pfs);
  P->x_words = o;
  P->lds = P->lds_h > P->lds_u ? P->lds_h : P->lds_u;
  if (P->lds_m > P->lds) P->lds = P->lds_m;
  return P->lds <= 160 * 1024;
}

// Fused Subscale WaveRNN 2x (Sec. 4.4) on the persistent kernel: the batch-1
// plan with 64 partial logits per head and half (high and low nibble of both
// sub-tensors' bytes) instead of 256.  Head fragments per wave: O1 [KH],
// O3 [KH] (block diagonal over the two quarters of a half), then the
// wave's class tile of O2 and of O4 over the head's KO column tiles.
WR_HD inline bool fused_plan(int H, PersistPlan* P) {
  if (!persist_plan(H, P)) return false;
  P->NM = P->mw_frags = P->lds_m = 0;             // no mirrors: single-buffered words
  P->x_hf = P->x_gfs = P->x_pfs = P->x_xcc = 0;
  wr_place(P, 0, 255);
  P->hw_frags = 2 * P->KH + 2 * P->KO;
  // head LDS: y_c and y_f operand images (KT fragments each), relu image (KO),
  // first-layer partials [2][64], misc [16], uniforms [2][64][8], targets [2][64][2]
  P->lds_h = (2 * P->KT + P->KO) * WR_FRAG + 4 * (2 * 64 + 16 + 2 * 64 * 8 + 2 * 64 * 2);
  int o = 0;
  auto take = [&](int n) { int r = o; o += wr_rup(n, WR_XALIGN); return r; };
  P->x_yc = take(P->Hh);
  P->x_yf = take(P->Hh);
  P->x_ga = take(3 * P->Hh);
  P->x_gf = take(3 * P->Hh);
  P->x_ps = 64;
  P->x_pc = take(P->NH * P->x_ps);
  P->x_pf = take(P->NH * P->x_ps);
  P->x_xcc = take(P->NH);
  P->x_words = o;
  P->lds = P->lds_h > P->lds_u ? P->lds_h : P->lds_u;
  return P->lds <= 160 * 1024;
}

// ---------------------------------------------------------------------------
// Block-sparse R (Sparse WaveRNN, Sec. 3.2) on the persistent kernel.
//
// Heads: split MLPs (heads j < NK hold 64-row slice j of O1 and the matching
// columns of O2; heads NK + j the same of O3, O4), NK = Hh / 64, and
// GU = ceil(Hh / 448) gate slots per preparing thread (GU > 1: gate state in
// LDS).
// Unit k owns the SR consecutive R rows SR k .. SR k + SR - 1 (row order
// g H + i, SR divides Hh, so a unit stays inside one gate and one half): BR =
// SR / BH block-rows of BH x BW blocks (4 x 4, or 16 x 1: 16 rows of one
// column).  Waves 0-3 compute: SL = 256 / SR consecutive lanes share a row.
// The kept blocks of a block-row in one half of the columns are dealt to the
// SL parts in turn (block i to part i mod SL), so lane (row, part) walks the
// same block list as the other rows of its block-row; each slot is one block:
// one u16 block-column index shared by the block-row's lanes of that part
// ([slot][BR][SL], the only index per kept block), and the lane's row of the
// block's weights (4 bf16 for 4 x 4, 1 for 16 x 1) in [slot][256 lanes].
// 16 x 1 slots go in quads, so one 8-byte read brings 4 weights or 4
// indices: weights [slot / 4][256][4], indices [slot / 4][BR][SL][4].
// Slots past a list's end hold zero weights.  Coarse-column slots come first,
// then fine.  Waves 4-7 read h from the heads and never store.
// ---------------------------------------------------------------------------
WR_HD inline bool sparse_plan(int H, int SR, int BH, int BW, int NRC, int NRF, PersistPlan* P) {
  if (H <= 0 || H % 128) return false;
  P->H = H;
  P->Hh = H / 2;
  P->KT = P->Hh / 32;
  P->RT = 4;
  P->HR = 64;
  P->KO = 2;
  const int KC = 2;
  P->KH = P->KT / KC;
  P->NK = P->Hh / P->HR;
  P->NH = 2 * P->NK;
  P->GU = (P->Hh + 447) / 448;
  if (P->NH > 32 || P->GU > 3) return false;
  if (SR < 16 || SR > 256 || 256 % SR || P->Hh % SR || NRC < 1 || NRF < 1) return false;
  if (!((BH == 4 && BW == 4) || (BH == 16 && BW == 1)) || SR % BH) return false;
  if (BW == 1) {   // 16 x 1: slots in quads (4 weights and 4 indices per read)
    NRC = (NRC + 3) / 4 * 4;
    NRF = (NRF + 3) / 4 * 4;
  }
  P->SR = SR;
  P->SL = 256 / SR;
  P->NRC = NRC;
  P->NRF = NRF;
  P->BH = BH;
  P->BW = BW;
  P->BR = SR / BH;
  P->UCT = 0;
  P->NCT = 3 * P->Hh / 16;
  P->NU = 3 * H / SR;
  P->NM = P->mw_frags = P->lds_m = 0;             // no mirrors: single-buffered words
  P->x_hf = P->x_gfs = P->x_pfs = P->x_xcc = 0;
  P->hw_frags = P->KH + 2 * P->KO;
  // head LDS: operand image (KT + KO fragments), first-layer partials
  // [KC][HR], logit sums [2][256], logits [256], then y [Hh] (GU = 1) or
  // h_c, h_f [2][Hh], prepared terms [5][Hh], fine words [4][Hh], I* [Hh][15]
  // (GU > 1), misc [16],
  // uniforms [2][64][2], targets [2][64]
  P->lds_h = (P->KT + P->KO) * WR_FRAG +
             4 * (KC * P->HR + 3 * 256 + (P->GU > 1 ? 26 * P->Hh : P->Hh) + 16 + 256 + 128);
  // unit LDS: block weights [NRC + NRF][256] (8 or 2 bytes each), block-column
  // indices [NRC + NRF][BR][SL] (u16), h [H], misc [16]
  P->u_wb = wr_rup((NRC + NRF) * 256 * (BW == 4 ? 8 : 2), 16);
  P->u_lds_w = P->u_wb + wr_rup((NRC + NRF) * P->BR * P->SL * 2, 16);
  P->lds_u = P->u_lds_w + 4 * (H + 16);
  wr_place(P, 0, 255);
  int o = 0;
  auto take = [&](int n) { int r = o; o += wr_rup(n, WR_XALIGN); return r; };
  P->x_yc = take(P->Hh);
  P->x_yf = take(P->Hh);
  P->x_ga = take(3 * P->Hh);
  P->x_gf = take(3 * P->Hh);
  P->x_ps = 256;
  P->x_pc = take(P->NK * P->x_ps);
  P->x_pf = take(P->NK * P->x_ps);
  P->x_xcc = take(P->NH);
  P->x_words = o;
  P->lds = P->lds_h > P->lds_u ? P->lds_h : P->lds_u;
  return P->lds <= 160 * 1024 && P->grid <= 256;
}

// ---------------------------------------------------------------------------
// Batched persistent kernel: G groups, each a copy of the batch-1 structure
// serving L vectors (independent utterances or subscale lanes) at once: as
// few per group as 8 groups allow (L = 2 up to 16 vectors, 4 up to 32, else 8),
// so each head reads and evaluates as few gate words as possible.  The MFMA operand A
// carries vector b in rows 2b (bf16 high part) and 2b+1 (remainder), so a
// group does the same number of matrix-core instructions as batch 1.
// Head j of group g sits at block 8j + g (one XCD per group); the units of all
// groups take the remaining blocks.  A unit owns UCT = 4 coarse and 4 fine
// row tiles: waves 0-3 the coarse tiles (coarse columns in LDS, fine columns
// in VGPRs), waves 4-7 the fine tiles (coarse columns in VGPRs, fine columns
// in LDS).
// ---------------------------------------------------------------------------
#define WR_BL 8           // most vectors per group
#define WR_BUCT 4         // coarse (and fine) row tiles per batched unit

struct BatchPlan {
  int H, Hh, KT, KH, NH, NCT, NU, G, grid;
  int L;                  // vectors per group (2, 4 or 8)
  int hw_frags;           // head fragments per wave (as the batch-1 plan)
  int u_lds_w;            // unit LDS weights: [UCT][KT] coarse tiles, then [UCT][KT] fine tiles
  int x_xcc;              // per group: the XCD of each head, published at the start
  int x_yc, x_yf, x_ga, x_gf, x_pc, x_pf, x_sp, x_xc, x_xf, x_cc, x_cf, x_words;   // per group: y [L][Hh],
      // g [3][Hh][L], p [NH][L][256], drawn samples [2][L], e-gate context terms [Hh][L] x 2,
      // drawn coarse and fine classes [L] each
  int KX;                 // subscale context column tiles (Dx / 32), 0 without context
  int HC;                 // drawn samples a unit keeps per utterance (ring, a power of two)
  int HS;                 // utterances whose samples a unit keeps (slots of HC)
  int RING;               // ints of LDS the sample rings take (0 with a context table)
  int SS;                 // slots of the drawn-sample words (a power of two >= 2 A + 2)
  int lds_h, lds_u, lds;
};

// Role of block b: head index j (group *g), NH + unit index, or -1 (idle).
WR_HD inline int wr_batch_role(const BatchPlan& P, int b, int* g) {
  if (b < 8 * P.NH && b % 8 < P.G) {
    *g = b % 8;
    return b / 8;
  }
  const int before = b < 8 * P.NH ? (b / 8) * P.G + (b % 8 < P.G ? b % 8 : P.G) : P.NH * P.G;
  const int ku = b - before;
  if (ku >= P.NU * P.G) return -1;
  *g = ku / P.NU;
  return P.NH + ku % P.NU;
}

// B, F, A: subscale factor, future horizon (F < 0: lockstep rows) and the
// steps A by which the units form the context ahead, which size the ring of
// drawn samples a unit keeps and the slots of the sample words.
WR_HD inline bool batch_plan(int H, int n_vectors, BatchPlan* P, int ctx_dim = 0, int B = 1, int F = -1,
                             int A = 0, bool table = false) {
  if (H <= 0 || H % 128 || n_vectors < 1 || n_vectors > 8 * WR_BL) return false;
  if (ctx_dim < 0 || ctx_dim % 32 || ctx_dim > 256 || B < 1 || F > 1024 || A < 0 || A > 3) return false;
  P->KX = ctx_dim / 32;
  P->H = H;
  P->Hh = H / 2;
  P->KT = P->Hh / 32;
  P->KH = P->KT / 2;
  P->NH = P->Hh / WR_HROWS;
  P->NCT = 3 * P->Hh / 16;
  if (P->NH > 7 || P->Hh > WR_THREADS - 64 || P->NCT % WR_BUCT) return false;
  P->NU = P->NCT / WR_BUCT;
  P->L = n_vectors <= 2 * WR_BL ? WR_BL / 4 : n_vectors <= 4 * WR_BL ? WR_BL / 2 : WR_BL;
  P->G = (n_vectors + P->L - 1) / P->L;
  int gr = 8 * (P->NH - 1) + P->G;           // the last head block + 1
  while (gr - P->NH * P->G < P->NU * P->G) ++gr;
  P->grid = gr;
  P->hw_frags = 2 * P->KH + 8;
  P->u_lds_w = 2 * WR_BUCT * P->KT * WR_FRAG;
  int o = 0;
  auto take = [&](int n) { int r = o; o += wr_rup(n, WR_XALIGN); return r; };
  P->x_yc = take(P->L * P->Hh);
  P->x_yf = take(P->L * P->Hh);
  P->x_ga = take(P->L * 3 * P->Hh);
  P->x_gf = take(P->L * 3 * P->Hh);
  P->x_pc = take(P->NH * P->L * 256);
  P->x_pf = take(P->NH * P->L * 256);
  P->SS = 2;
  while (P->SS < 2 * A + 2) P->SS *= 2;
  P->x_sp = take(P->SS * P->L);
  P->x_xc = take(P->L * P->Hh);
  P->x_xf = take(P->L * P->Hh);
  P->x_cc = take(P->L);
  P->x_cf = take(P->L);
  P->x_xcc = take(P->NH);
  P->x_words = o;
  // head: operand images (2 KT + 2 fragments), first-layer partials [2][L][64],
  // logit sums [L][256], logits [L][256], both halves of h and the staged
  // gate inputs [2 + 4][L][448], bias row offsets [L], misc [64],
  // uniforms [2][L][64][2], targets [2][L][64], and with up to 4 vectors the
  // fine half's staged gate inputs [4][L][448]
  P->lds_h = (2 * P->KT + 2) * WR_FRAG + 4 * (2 * P->L * 64 + 2 * P->L * 256 + 6 * P->L * 448 + 2 * P->L + 64 +
                                               2 * P->L * 64 * 2 + 2 * P->L * 64 + (P->L <= 4 ? 4 * P->L * 448 : 0));
  // Ring of drawn samples per utterance: lockstep, the Dx/2 samples before
  // a row plus the row; with horizon F the lanes of an utterance are up to
  // (B - 1)(F + 1 + A) positions apart, so the newest sample and the oldest
  // one a context still reads are at most B (B - 1)(F + 1 + A) + Dx/4 apart.
  // (With a context table, read from HBM at each step, there is no ring.)
  {
    const int need = F < 0 ? ctx_dim / 2 + 2 * B : B * (B - 1) * (F + 1 + A) + ctx_dim / 2 + B;
    P->HC = 256;
    while (!table && P->HC < need) P->HC *= 2;
    P->HS = (ctx_dim > 0 && P->L > B) ? P->L / B : 1;
    P->RING = ctx_dim > 0 && !table ? P->HS * P->HC : 0;
  }
  // unit: weights, operand image (2 KT fragments), context image (KX fragments),
  // sample rings [HS][HC], misc [16]
  P->lds_u = P->u_lds_w + (2 * P->KT + P->KX) * WR_FRAG + 4 * (P->RING + 16);
  P->lds = P->lds_h > P->lds_u ? P->lds_h : P->lds_u;
  return P->lds <= 160 * 1024 && P->grid <= 256;
}
