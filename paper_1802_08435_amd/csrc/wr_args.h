// Kernel argument blocks of libwavernn (shared by the host launcher and kernels).
#pragma once
#include <stdint.h>
#include "wr_layout.h"

typedef unsigned long long u64;
typedef uint32_t xw;        // exchange word (value with the step parity in its lowest bit)

#define WR_TRACE_SLOTS 32   // per traced step: timestamps (100 MHz) of phase ends

struct SmallArgs {
  const float* image;        // packed fp32 weights, SmallLayout order
  const float* Wc;           // [3H][Dc] or null
  const float* feat;         // [S][n_frames][Dc] or null
  int64_t n_frames;
  int H, Dc, frame_len;
  int64_t T, t0;
  uint64_t seed;
  const uint16_t* target;    // [S][T] or null (free sampling)
  uint16_t* out;             // [S][T] or null
  float* zc_out;             // [S][T][256] or null
  float* zf_out;
  float* nll_out;            // [S][T] or null
  const float* h_in;         // [S][H] or null
  const uint8_t* c_in;
  const uint8_t* f_in;
  float* h_out;              // or null
  uint8_t* c_out;
  uint8_t* f_out;
};

struct PersistArgs {
  PersistPlan P;
  const uint4* hw;          // [NH][8 waves][hw_frags][64 lanes] head fragments
  const uint4* uw;          // [NU] unit LDS blocks of P.u_lds_w bytes
  const uint4* ur;          // [2][NU*UCT][KT][64] coarse, then fine tiles x fine columns (VGPR-resident)
  const uint4* mw;          // [NM][8 waves][mw_frags][64 lanes] mirror fragments, or null (no mirrors)
  const float* Iw;          // [3H][3], I* mask applied
  const float* b1;          // [Hh]
  const float* b2;          // [256]
  const float* b3;
  const float* b4;
  const float* cb;          // [n_cb][3H] gate bias + conditioning per frame
  int64_t n_cb;
  int frame_len;
  int64_t T, t0;
  uint64_t seed, stream_id;
  const uint16_t* target;   // [T] or null
  uint16_t* out;            // [T] or null
  float* zc_out;            // [T][256] or null
  float* zf_out;
  float* nll_out;           // [T] or null
  const float* h_in;        // [H] or null
  const uint8_t* c_in;
  const uint8_t* f_in;
  float* h_out;
  uint8_t* c_out;
  uint8_t* f_out;
  xw* xc;                   // exchange words (wr_device.h), zeroed before the launch
  unsigned* err;
  u64 limit;                // wait limit in 100 MHz ticks
  u64* trace;               // [trace_steps][WR_TRACE_SLOTS] phase timestamps or null
  int64_t trace_steps;
  int F;                    // fused 2x model: future horizon (sub-tensor 1 runs F + 1 steps behind)
  int64_t rows;             // fused 2x model: positions per sub-tensor (samples / 2)
};

// Teacher-forced recurrence of the dense batch-1 model (wr_score.hip).
// With several utterances (wr_score_multi, nv of them) every per-utterance
// array holds them one after another: cb [nv][n_cb][3H], target [nv][T],
// h [nv][H], c / f [nv], traj [nv][T][Hh]; xc is [2][8][H].
struct ScoreArgs {
  const uint4* w;           // [H/16][3][H/32][64 lanes] R fragments: workgroup k, gate g: rows g H + 16 k ..
  const float* Iw;          // [3H][3], I* mask applied
  const float* cb;          // [n_cb][3H] gate bias + conditioning per frame
  int64_t n_cb;
  int frame_len;
  int H, Hh;
  int64_t T, t0;
  const uint16_t* target;   // [T]
  const float* h_in;        // [H] or null
  const uint8_t* c_in;
  const uint8_t* f_in;
  float* h_out;             // [H] or null
  uint8_t* c_out;
  uint8_t* f_out;
  float* traj_c;            // [T][Hh] coarse half of h after each step
  float* traj_f;            // [T][Hh] fine half
  xw* xc;                   // [2][H] exchange words, zeroed before the launch
  unsigned* err;
  u64 limit;
  int nv;                   // wr_score_multi: utterances of the launch (1..8)
};

struct BatchArgs {
  BatchPlan P;
  const uint4* hw;          // [NH][8 waves][hw_frags][64 lanes] head fragments (as PersistArgs::hw)
  const uint4* uw;          // [NU] unit LDS blocks of P.u_lds_w bytes
  const uint4* ur;          // [NU][8 waves][KT][64] VGPR-resident unit fragments
  const float* Iw;          // [3H][3], I* mask applied
  const float* b1;          // [Hh]
  const float* b2;          // [256]
  const float* b3;
  const float* b4;
  const uint4* ux;          // [NU][8 waves][KX][64] context-projection fragments (subscale) or null
  const float* ctab;        // horizon schedule only: context table [S][ctab_rows][Dx], or null (window
                            // context); vector v = lane s at position p reads row
                            // p - (ctab_row0 + s ctab_step) of its block
  int64_t ctab_rows, ctab_row0, ctab_step;
  const float* cb;          // [U][n_cb][3H] gate bias + conditioning per utterance and frame
  int64_t n_cb;
  int frame_len;
  int S;                    // vectors in use (the last group may be partly idle)
  int B;                    // subscale factor: vector v is lane v % B of utterance v / B (1: plain)
  int F;                    // subscale future horizon (Sec. 4.2): lane s runs position t - s (F + 1 + A)
                            // at step t; < 0: lockstep rows (position t)
  int A;                    // steps by which the units form a horizon context ahead (0: at the step before)
  int64_t rows;             // positions per lane (samples per utterance / B)
  int64_t T, t0;            // steps of this launch and its first absolute step (with a horizon: the
                            // first step of the schedule; lockstep rows: the first row)
  uint64_t seed;
  const uint16_t* target;   // [U][B rows] samples in time order, or null
  uint16_t* out;            // [U][B rows] (with a horizon; lockstep rows: from row t0 on, utterances
                            // B rows apart) or null
  const uint16_t* prev;     // window context, t0 > 0: the utterances' samples [U][B rows] made before
                            // step t0, which start the units' rings; null otherwise
  float* zc_out;            // [U][B T][256] or null
  float* zf_out;
  float* nll_out;           // [U][B T] or null
  const float* h_in;        // [S][H] or null
  const uint8_t* c_in;      // [S]
  const uint8_t* f_in;
  float* h_out;
  uint8_t* c_out;
  uint8_t* f_out;
  xw* xc;                   // [G][P.x_words] exchange words, zeroed before the launch
  unsigned* err;
  u64 limit;
  u64* trace;               // [trace_steps][WR_TRACE_SLOTS] (group 0) or null
  int64_t trace_steps;
};

// One GEMM of the conditioning CNN: dst[m][n] (epilogue) over
// acc = sum_k A[m][k] W[n][k], n < N, on 128 x 128 tiles.
#define WR_CNN_MAXB 64   // sub-tensors of a streamed CNN run at most
struct CnnGemmArgs {
  const float* src;       // activations [M][kin]
  int kin;                // source row width (a multiple of 32)
  int taps, dil;          // A row m = [src row m + tap dil (same block, tap < taps)], zero past the block
                          // and past the utterance's last row
  int rows;               // rows per block (one utterance's sub-tensor, or its window)
  int B;                  // blocks per utterance (sub-tensors): block (u, s) = m / rows
  int64_t row0, row_step, rows_utt;   // row k of block (u, s) is utterance row row0 + s row_step + k,
                                      // of rows_utt
  int M;                  // activation rows
  int K;                  // taps x kin
  const uint4* w;         // weight fragments [N / 16][K / 32] x 64 lanes
  const float* bias;      // [N]
  int N;                  // a multiple of 128
  float* dst;             // [M][N] rows, or with out_B > B block (u, s) of the run at block u out_B + out_s0 + s
  int out_B, out_s0;      // (out_B = B, out_s0 = 0: row m at row m)
  int epi;                // 0: acc + bias; 1: relu(acc + bias); 2: dst + (acc + bias)
  int group;              // K-steps per accumulation group (the sum is ((g0 + g1) + g2) + ..., each g_q from 0)
  int split;              // 1: a workgroup runs every group of its tile; > 1 (= the number of groups):
                          // workgroup (tile, q) writes g_q to part[q] and wr_cnn_reduce adds them in order
  float* part;            // [groups][M][N] (split > 1)
  int tiles_m, tiles, per_xcd;   // 128-row tiles, all tiles, tiles x split per XCD slot
  // Streamed runs (rng = 1): block b of the run is (utterance b / B, sub-tensor out_s0 + b % B); its
  // row k is utterance row lo[s] + k, and only rows below hi[s] are computed (the others are read as
  // zero and not stored).  With src_abs (dst_abs) the source (destination) is a whole-utterance array
  // [U][out_B][rows_utt][width] at that row (taps past rows_utt read zero); otherwise it is indexed by
  // the run's row m.
  int rng, src_abs, dst_abs;
  int lo[WR_CNN_MAXB], hi[WR_CNN_MAXB];
};
#define CNN_TM 128
#define CNN_TN 128
#define CNN_THREADS 512
#define CNN_LDS_BUF (3 * 8 * 1024)   // A high, A low (8 row tiles each), W (8 column tiles), fragments of 1 KiB

// Input rows of the conditioning CNN (see wr_cnn_input).
struct CnnInputArgs {
  const uint16_t* seq;    // [U][n_samples] samples in time order
  int64_t n_samples;
  int B;
  int64_t rows;           // rows of the utterance (n_samples / B)
  int win;                // rows per (utterance, sub-tensor) block
  int64_t row0, row_step; // block (u, s) covers utterance rows row0 + s row_step ...
  int64_t front0, front_step;   // sub-tensor z has made rows up to front0 + z front_step
  int s0, nsb;            // the run covers sub-tensors s0 .. s0 + nsb - 1 of each utterance: block m / win =
                          // (u, s - s0)
  int M, kin;
  float* x;               // [M][kin]
  int rng;                // streamed run: block (u, s - s0)'s row k is utterance row lo[s] + k
  int lo[WR_CNN_MAXB];
};

// Kernel entry points (taken by address in the launcher).
const void* wr_small_kernel_ptr();
const void* wr_uniforms_kernel_ptr();
const void* wr_persist_kernel_ptr(int KH);   // null if no instantiation for KH
const void* wr_score_kernel_ptr(int KT2);    // teacher-forced recurrence for H = 32 KT2; null if none
const void* wr_score_multi_ptr(int KT2);     // the same for up to 8 utterances at once
const void* wr_score_nll_ptr();
const void* wr_sparse_kernel_ptr(int KH, int GU);   // null if no instantiation
const void* wr_cond_kernel_ptr();
const void* wr_batch_kernel_ptr(int KH, bool ctx, int L, bool lag);   // null if no instantiation (KH, L vectors
                                                                      // per group, lag: a future-horizon schedule)
const void* wr_batch_floor_kernel_ptr(int KH, bool ctx, int L, bool lag);   // null if no instantiation
const void* wr_fill_kernel_ptr();
const void* wr_fused_kernel_ptr(int KH);     // null if no instantiation
const void* wr_floor_kernel_ptr();
const void* wr_cnn_gemm_ptr();
const void* wr_cnn_input_ptr();
const void* wr_cnn_reduce_ptr();
