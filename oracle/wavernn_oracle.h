/*
 * WaveRNN oracle (test infrastructure only) -- C interface used via ctypes by
 * the tests, the smoke check and the benchmark's CPU baseline.
 * See wavernn_oracle.c for what is computed and the readings of the paper.
 */
#ifndef WAVERNN_ORACLE_H
#define WAVERNN_ORACLE_H
#include <stdint.h>

#define ORC_MAX_CLASSES 256   /* 8-bit coarse / fine softmax (Sec. 2) */
#define ORC_MAX_HIDDEN 4096

/* Subscale conditioning network (Sec. 4.1, 5); readings in wavernn_oracle.c.
 *   Win [Rc][2B] bin [Rc]; Wc [layers][Cc][3][Rc] bc [layers][Cc] (taps at rows
 *   k, k + d, k + 2d, d = 2^(l mod 5)); Wo [layers][Rc][Cc] bo [layers][Rc];
 *   Wp [Dx][Rc] bp [Dx].  The paper: 10 layers, Cc = 384, Rc = 768. */
typedef struct {
  int32_t B, Rc, Cc, Dx, layers;
  const float *Win, *bin, *Wc, *bc, *Wo, *bo, *Wp, *bp;
} orc_cnn;

/* All matrices fp32 row-major.  Gate order u, r, e.
 *   R  [3][H][H]      recurrent matrix (Eq. 2); zeroed entries = pruned weights
 *   I  [3][H][3]      input matrix, columns (c_{t-1}, f_{t-1}, c_t); column 2 of
 *                     rows i < H/2 is ignored (the I* mask)
 *   b  [3][H]         gate biases
 *   Wc [3H][Dc]       conditioning projection (Dc = 0: none)
 *   Wx [3H][Dx]       subscale context projection (Dx = 0: none)
 *   O1 [H/2][H/2] b1 [H/2]   O2 [256][H/2] b2 [256]   (coarse head)
 *   O3 [H/2][H/2] b3 [H/2]   O4 [256][H/2] b4 [256]   (fine head)
 *   cnn               optional conditioning network of a subscale model with F >= 0 */
typedef struct {
  int32_t H, Dc, frame_len, B, Dx;
  int32_t F;   /* subscale future horizon (Sec. 4.2): < 0 lockstep rows, >= 0 the paper's order */
  const float *R, *I, *b, *Wc, *Wx;
  const float *O1, *b1, *O2, *b2, *O3, *b3, *O4, *b4;
  const orc_cnn* cnn;   /* with F >= 0: the context of sub-tensor s is this network's output (NULL: window) */
} orc_model;

float orc_exp(float y);
float orc_sigmoid(float x);
float orc_tanh(float x);
float orc_scale(int v);
void orc_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);
void orc_uniforms(uint64_t seed, uint64_t stream, int64_t t, float* uc, float* uf);
int orc_draw(const float* z, int n, float u);

/* Subscale context of sample n = B*i + s of an utterance of N samples whose
 * samples so far are seq[N] (Dx/2 (c, f) pairs into ctx[Dx]); the rule of
 * the model (lockstep for F < 0, future horizon F otherwise). */
void orc_subscale_context(const orc_model* m, const uint16_t* seq, int64_t N, int32_t s, int64_t i, float* ctx);

/* Runs S utterances of T samples (B = 1: starting at absolute sample t0).
 * feat [S][n_frames][Dc]; target [S][T] (NULL: sample freely); state h [S*B][H],
 * cprev/fprev [S*B] are read and updated; out [S][T] (16-bit, 256*c + f);
 * zc/zf [S][T][256] logits and nll [S][T] (nats) are optional.  Returns 0 or -1. */
int orc_run(const orc_model* m, int32_t S, int64_t T, int64_t t0, const float* feat, int64_t n_frames,
            uint64_t seed, const uint16_t* target, float* h, uint8_t* cprev, uint8_t* fprev, uint16_t* out,
            float* zc, float* zf, double* nll);
/* orc_run teacher-forced on the lanes (sub-tensors) [lane_lo, lane_hi) of every
 * utterance only (with a target the lanes are independent); the outputs of
 * the other lanes are left as they were.  Returns 0 or -1. */
int orc_run_lanes(const orc_model* m, int32_t S, int64_t T, const float* feat, int64_t n_frames,
                  const uint16_t* target, float* h, uint8_t* cprev, uint8_t* fprev, float* zc, float* zf,
                  double* nll, int32_t lane_lo, int32_t lane_hi);
/* Fused Subscale WaveRNN 2x (Sec. 4.4); readings in wavernn_oracle.c.  Q = H/4.
 *   R  [3][H][H]       one recurrent matrix over the whole state
 *   I  [3][H][6]       columns (c0, f0, c1, f1) of each sub-tensor's last sample,
 *                      then c0_t, c1_t; coarse units [0, 2Q) use the first four,
 *                      fine units of sub-tensor s those and the column of c_s,t
 *   b  [3][H]          gate biases;  Wc [3H][Dc] conditioning (Dc = 0: none)
 *   O1 [4][Q][Q] b1 [4][Q]          head k = 2 level + s (level 0 coarse, 1 fine)
 *   O2 [4][2][16][Q] b2 [4][2][16]  [k][0] high nibble, [k][1] low nibble   */
typedef struct {
  int32_t H, F, Dc, frame_len;
  const float *R, *I, *b, *Wc, *O1, *b1, *O2, *b2;
} orc_fused_model;

/* Runs S utterances of N samples (N even) from h = 0 and last samples
 * (128, 0): N/2 + F + 1 steps.  feat [S][n_frames][Dc]; target [S][N] (NULL:
 * sample freely); out [S][N]; zc/zf [S][N][32] (high then low nibble logits),
 * nll [S][N] (nats, four nibbles) and h_final [S][H] are optional.  Returns 0
 * or -1. */
int orc_fused_run(const orc_fused_model* m, int32_t S, int64_t N, const float* feat, int64_t n_frames,
                  uint64_t seed, const uint16_t* target, uint16_t* out, float* zc, float* zf, double* nll,
                  float* h_final);
/* Conditioning vectors out [N/B][Dx] of sub-tensor s of one utterance whose
 * samples are seq [N] (N a multiple of B).  Returns 0 or -1. */
int orc_ctx_cnn(const orc_cnn* m, const uint16_t* seq, int64_t N, int32_t s, float* out);
#endif
