/*
 * WaveRNN oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, scalar CPU implementation of the WaveRNN sampling step of
 * "Efficient Neural Audio Synthesis" (Kalchbrenner et al., 2018), used to check
 * the GPU library.  Only the tests, the smoke check and the benchmark's CPU
 * baseline may load it; the GPU library neither links nor calls it, and it shares
 * no code with the GPU library.
 *
 * What it computes (per stream, per step t):
 *   x_t = [c_{t-1}, f_{t-1}, c_t], each byte scaled from [0,255] to [-1,1]   (Sec. 2, text after Eq. 2)
 *   u = sigma(R_u h + I*_u x + b_u),  r = sigma(R_r h + I*_r x + b_r)        (Eq. 2)
 *   e = tanh(r o (R_e h) + I*_e x + b_e),  h' = u o h + (1-u) o e            (Eq. 2)
 *   y_c, y_f = split(h');  P(c) = softmax(O2 relu(O1 y_c + b1) + b2)         (Eq. 2)
 *                          P(f) = softmax(O4 relu(O3 y_f + b3) + b4)
 *   I* is masked: c_t reaches only the fine half of u, r, e                  (Sec. 2, text after Eq. 2)
 *   gates of the coarse half are evaluated first, c_t is sampled, then the
 *   fine half is evaluated and f_t is sampled                                (Fig. 1 caption)
 *
 * Precision: weights and activations are fp32 (weights may carry values rounded
 * to bf16 by the caller); the paper keeps activations and arithmetic in 32-bit
 * float (Sec. 3.3).  Readings of the paper fixed here (the paper is silent):
 *   - every dot product is a chain of fused multiply-adds in increasing index
 *     order starting from +0;
 *   - one bias per gate, added outside the reset product; biases on O1..O4;
 *   - exp is evaluated by Cody-Waite range reduction and a degree-7 Taylor
 *     polynomial (Cody & Waite, 1980), sigma(x) = 1/(1+exp(-x)),
 *     tanh(x) = sign(x)(1-q)/(1+q) with q = exp(-2|x|);
 *   - a class is drawn by inverse CDF: k* = #{k : C_k <= U*C_255} over the
 *     running sums C_k of exp(z_k - max z), clamped to the last class with
 *     nonzero weight;
 *   - uniforms come from Philox4x64-10 (Salmon et al., SC'11) with key
 *     (seed, 0) and counter (t, stream, 0, 0); U = (word >> 40) * 2^-24,
 *     word 0 for the coarse draw and word 1 for the fine draw;
 *   - initial state h = 0, c_{-1} = 128, f_{-1} = 0 unless given;
 *   - conditioning: a feature frame of Dc values per frame_len samples enters
 *     every gate pre-activation through W_cond (3H x Dc);
 *   - Subscale (Sec. 4, Eq. 4): sub-tensor s holds the samples n = B*i + s,
 *     i = 0 .. N/B - 1, generated from its own state (lane s); a context of
 *     Dx/2 samples, each as (c, f) scaled, enters the gates through W_ctx
 *     (3H x Dx).  Two readings:
 *       F < 0, lockstep rows: all B lanes make row i together; the context of
 *         n is the Dx/2 samples before n, zero for those of row i or later;
 *       F >= 0, the paper's order with future horizon F (Sec. 4.2): sub-tensor
 *         s is generated after sub-tensors 0 .. s-1; the context of sample
 *         B*i + s holds the samples of the previous sub-tensors z < s up to
 *         position i + F (Sec. 4.1: the conditioning sees the previous
 *         sub-tensors; its own sub-tensor reaches the sample through the
 *         recurrent state and inputs; no distant dependencies, Sec. 4.3), as
 *         the Dx/4 samples before n and the Dx/4 after n, zero where not seen.
 *         Generated here sub-tensor by sub-tensor, in the paper's order.
 *       With a conditioning network attached (F >= 0), the context of sample
 *         B*i + s is row i of orc_ctx_cnn for sub-tensor s, computed once the
 *         sub-tensors before s are complete (Sec. 4.1: each sub-tensor is
 *         generated conditioned on the previous ones through the CNN).
 *   - Fused Subscale WaveRNN 2x (Sec. 4.4): orc_fused_run, and the masked
 *     dilated CNN that conditions the Subscale WaveRNN (Sec. 4.1, 5):
 *     orc_ctx_cnn, each with its own readings in its section below.
 *
 * Build: cc -O2 -ffp-contract=off -fPIC -shared (no fast-math; fmaf only where written).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "wavernn_oracle.h"

/* ------------------------------------------------------------------------- */
/* Elementary functions (reading: Cody-Waite + Taylor, see header comment)    */
/* ------------------------------------------------------------------------- */

static float g_ln2_hi, g_ln2_lo, g_log2e, g_inv_fact[8];
static int g_consts_ready = 0;

/* ln 2 split into a 15-significant-bit head (so k*ln2_hi is exact for |k| < 512)
 * and a tail, both derived here from the double-precision value of ln 2;
 * Taylor coefficients 1/i! rounded to fp32. */
static void init_consts(void) {
  if (g_consts_ready) return;
  double ln2 = log(2.0);
  int e;
  double m = frexp(ln2, &e);                   /* ln2 = m * 2^e, m in [0.5,1) */
  double head = ldexp(floor(ldexp(m, 15)), e - 15);
  g_ln2_hi = (float)head;
  g_ln2_lo = (float)(ln2 - head);
  g_log2e = (float)(1.0 / ln2);
  double f = 1.0;
  for (int i = 0; i < 8; ++i) {
    if (i > 0) f *= i;
    g_inv_fact[i] = (float)(1.0 / f);
  }
  g_consts_ready = 1;
}

float orc_exp(float y) {
  init_consts();
  if (y != y) return y;
  if (y < -86.0f) return 0.0f;           /* result would be below 2^-124 */
  if (y > 88.0f) return INFINITY;
  float k = rintf(y * g_log2e);          /* nearest integer, ties to even */
  float r = fmaf(-k, g_ln2_hi, y);
  r = fmaf(-k, g_ln2_lo, r);
  float p = g_inv_fact[7];
  for (int i = 6; i >= 0; --i) p = fmaf(p, r, g_inv_fact[i]);
  int ki = (int)k;                       /* in [-124, 127] */
  uint32_t bits = (uint32_t)(ki + 127) << 23;
  float two_k;
  memcpy(&two_k, &bits, 4);
  return p * two_k;
}

float orc_sigmoid(float x) { return 1.0f / (1.0f + orc_exp(-x)); }

float orc_tanh(float x) {
  float a = fabsf(x);
  float q = orc_exp(-2.0f * a);
  float t = (1.0f - q) / (1.0f + q);
  return copysignf(t, x);
}

static float relu(float v) { return v > 0.0f ? v : 0.0f; }

/* Byte -> [-1, 1]: (2v - 255) / 255, correctly rounded (Sec. 2: scalars in
 * [0,255] scaled to [-1,1]). */
float orc_scale(int v) { return (float)(2 * v - 255) / 255.0f; }

/* Dot product as an fma chain in increasing index order from +0. */
static float dot(const float* w, const float* x, int n) {
  float acc = 0.0f;
  for (int j = 0; j < n; ++j) acc = fmaf(w[j], x[j], acc);
  return acc;
}

/* ------------------------------------------------------------------------- */
/* Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11)                          */
/* ------------------------------------------------------------------------- */

static void mulhilo64(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
  unsigned __int128 p = (unsigned __int128)a * b;
  *hi = (uint64_t)(p >> 64);
  *lo = (uint64_t)p;
}

void orc_philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ULL, M1 = 0xCA5A826395121157ULL;
  const uint64_t W0 = 0x9E3779B97F4A7C15ULL, W1 = 0xBB67AE8584CAA73BULL;
  uint64_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint64_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) { k0 += W0; k1 += W1; }
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo64(M0, c[0], &hi0, &lo0);
    mulhilo64(M1, c[2], &hi1, &lo1);
    uint64_t n0 = hi1 ^ c[1] ^ k0, n1 = lo1, n2 = hi0 ^ c[3] ^ k1, n3 = lo0;
    c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
  }
  memcpy(out, c, sizeof c);
}

void orc_uniforms(uint64_t seed, uint64_t stream, int64_t t, float* uc, float* uf) {
  uint64_t ctr[4] = {(uint64_t)t, stream, 0, 0}, key[2] = {seed, 0}, w[4];
  orc_philox4x64_10(ctr, key, w);
  *uc = (float)(w[0] >> 40) * (1.0f / 16777216.0f);
  *uf = (float)(w[1] >> 40) * (1.0f / 16777216.0f);
}

/* ------------------------------------------------------------------------- */
/* Softmax sampling (Eq. 2 softmax; inverse CDF reading)                       */
/* ------------------------------------------------------------------------- */

int orc_draw(const float* z, int n, float u) {
  float m = z[0];
  for (int k = 1; k < n; ++k) if (z[k] > m) m = z[k];
  float w[ORC_MAX_CLASSES], c[ORC_MAX_CLASSES];
  float run = 0.0f;
  for (int k = 0; k < n; ++k) {
    w[k] = orc_exp(z[k] - m);
    run = run + w[k];
    c[k] = run;
  }
  float thr = u * c[n - 1];
  int count = 0;
  for (int k = 0; k < n; ++k) count += (c[k] <= thr);
  if (count == n) {
    count = n - 1;
    while (count > 0 && !(w[count] > 0.0f)) --count;
  }
  return count;
}

/* -log softmax(z)[k] in double from fp32 logits (plain definition). */
static double neg_log_prob(const float* z, int n, int k) {
  double m = z[0];
  for (int j = 1; j < n; ++j) if (z[j] > m) m = z[j];
  double s = 0.0;
  for (int j = 0; j < n; ++j) s += exp((double)z[j] - m);
  return -(((double)z[k] - m) - log(s));
}

/* ------------------------------------------------------------------------- */
/* The recurrent step                                                         */
/* ------------------------------------------------------------------------- */

/* Additive gate term that does not depend on h or x: bias + conditioning
 * (+ subscale context).  add[g*H + i] for gate g in {u, r, e}. */
static void gate_additive(const orc_model* m, const float* feat_frame, const float* ctx, float* add) {
  const int H = m->H;
  for (int row = 0; row < 3 * H; ++row) {
    float a = m->b[row];
    if (m->Dc > 0) a = dot(m->Wc + (size_t)row * m->Dc, feat_frame, m->Dc) + m->b[row];
    if (m->Dx > 0) a = a + dot(m->Wx + (size_t)row * m->Dx, ctx, m->Dx);
    add[row] = a;
  }
}

/* Gates for units i in [lo, hi): Eq. 2 with the masked input matrix.
 * x has three entries; for the coarse half (i < H/2) the third is ignored. */
static void gru_units(const orc_model* m, const float* G, const float* add, const float* x,
                      const float* h_prev, float* h_new, int lo, int hi) {
  const int H = m->H, Hh = H / 2;
  for (int i = lo; i < hi; ++i) {
    float ix[3];
    for (int g = 0; g < 3; ++g) {
      const float* Ig = m->I + ((size_t)g * H + i) * 3;
      ix[g] = dot(Ig, x, i < Hh ? 2 : 3);
    }
    float au = G[0 * H + i] + (ix[0] + add[0 * H + i]);
    float ar = G[1 * H + i] + (ix[1] + add[1 * H + i]);
    float u = orc_sigmoid(au);
    float r = orc_sigmoid(ar);
    float e = orc_tanh(fmaf(r, G[2 * H + i], ix[2] + add[2 * H + i]));
    h_new[i] = fmaf(u, h_prev[i], (1.0f - u) * e);
  }
}

/* One output head: z = Ob relu(Oa y + ba) + bb (Eq. 2). */
static void head(const orc_model* m, const float* Oa, const float* ba, const float* Ob, const float* bb,
                 const float* y, float* z) {
  const int Hh = m->H / 2;
  float hid[ORC_MAX_HIDDEN / 2];
  for (int k = 0; k < Hh; ++k) hid[k] = relu(dot(Oa + (size_t)k * Hh, y, Hh) + ba[k]);
  for (int v = 0; v < ORC_MAX_CLASSES; ++v) z[v] = dot(Ob + (size_t)v * Hh, hid, Hh) + bb[v];
}

/* Whether sample q = B*k + z of an utterance of N samples is in the context
 * of sample B*i + s under the future-horizon rule. */
static int seen_lagged(int B, int F, int64_t N, int32_t s, int64_t i, int64_t q) {
  if (q < 0 || q >= N) return 0;
  const int64_t k = q / B, z = q % B;
  return z < s && k <= i + F;
}

void orc_subscale_context(const orc_model* m, const uint16_t* seq, int64_t N, int32_t s, int64_t i, float* ctx) {
  const int B = m->B, P = m->Dx / 2;
  const int64_t n = (int64_t)B * i + s;
  for (int j = 0; j < P; ++j) {
    int64_t q;
    int seen;
    if (m->F < 0) {                 /* lockstep: the samples before n made before row i */
      q = n - 1 - j;
      seen = q >= 0 && q < (int64_t)B * i;
    } else {                        /* horizon F: Dx/4 samples before n, then Dx/4 after */
      q = j < P / 2 ? n - 1 - j : n + 1 + (j - P / 2);
      seen = seen_lagged(B, m->F, N, s, i, q);
    }
    ctx[2 * j] = seen ? orc_scale(seq[q] >> 8) : 0.0f;
    ctx[2 * j + 1] = seen ? orc_scale(seq[q] & 255) : 0.0f;
  }
}

/* Lanes [lane_lo, lane_hi) of every utterance; the others are skipped (teacher forcing only). */
static int run_lanes(const orc_model* m, int32_t S, int64_t T, int64_t t0, const float* feat, int64_t n_frames,
                     uint64_t seed, const uint16_t* target, float* h, uint8_t* cprev, uint8_t* fprev, uint16_t* out,
                     float* zc_out, float* zf_out, double* nll_out, int32_t lane_lo, int32_t lane_hi) {
  const int H = m->H, Hh = H / 2, B = m->B > 0 ? m->B : 1;
  if (H <= 0 || (H & 1) || H > ORC_MAX_HIDDEN || S <= 0 || T < 0) return -1;
  if (lane_lo < 0 || lane_hi > B || lane_lo >= lane_hi || ((lane_lo > 0 || lane_hi < B) && target == NULL)) return -1;
  if (B > 1 && (T % B != 0 || t0 != 0)) return -1;
  if (m->Dc > 0 && (m->frame_len <= 0 || feat == NULL)) return -1;
  if (m->Dx > 0 && (B == 1 || m->Dx % (m->F < 0 ? 2 : 4) != 0)) return -1;
  if (m->cnn && (m->F < 0 || m->cnn->B != B || m->cnn->Dx != m->Dx)) return -1;
  if (target == NULL && out == NULL) return -1;
  if (T == 0) return 0;
  float* G = (float*)malloc(sizeof(float) * 3 * H);
  float* add = (float*)malloc(sizeof(float) * 3 * H);
  float* hn = (float*)malloc(sizeof(float) * H);
  float* ctx = (float*)malloc(sizeof(float) * (m->Dx > 0 ? m->Dx : 1));
  float zc[ORC_MAX_CLASSES], zf[ORC_MAX_CLASSES];
  const int64_t rows = T / B;
  float* ctab = m->cnn ? (float*)malloc(sizeof(float) * (size_t)(rows > 0 ? rows : 1) * m->Dx) : NULL;
  /* lockstep: row by row, lane by lane; horizon F: lane (sub-tensor) by lane */
  const int lagged = B > 1 && m->F >= 0;
  const int64_t n_outer = lagged ? B : rows, n_inner = lagged ? rows : B;
  for (int32_t s = 0; s < S; ++s) {
    uint16_t* seq = out ? out + (size_t)s * T : NULL;   /* samples of utterance s, time order */
    const uint16_t* tgt = target ? target + (size_t)s * T : NULL;
    for (int64_t o = 0; o < n_outer; ++o) {
      if (lagged && (o < lane_lo || o >= lane_hi)) continue;
      /* conditioning CNN: sub-tensor o's context rows from the finished sub-tensors before it */
      if (m->cnn) orc_ctx_cnn(m->cnn, tgt ? tgt : seq, T, (int32_t)o, ctab);
      for (int64_t in = 0; in < n_inner; ++in) {
        const int64_t i = lagged ? in : o;
        const int lane = (int)(lagged ? o : in);
        if (lane < lane_lo || lane >= lane_hi) continue;
        const int64_t st = (int64_t)s * B + lane;   /* state / Philox stream index */
        const int64_t n = (B == 1) ? t0 + i : B * i + lane; /* absolute sample index */
        const int64_t local = (B == 1) ? i : n;             /* index into this call's arrays */
        float* hs = h + (size_t)st * H;
        const float* frame = NULL;
        if (m->Dc > 0) {
          int64_t fr = n / m->frame_len;
          if (fr >= n_frames) fr = n_frames - 1;
          frame = feat + ((size_t)s * n_frames + fr) * m->Dc;
        }
        if (m->cnn) memcpy(ctx, ctab + (size_t)i * m->Dx, sizeof(float) * m->Dx);
        else if (m->Dx > 0) orc_subscale_context(m, tgt ? tgt : seq, T, lane, i, ctx);
        gate_additive(m, frame, ctx, add);
        for (int row = 0; row < 3 * H; ++row) G[row] = dot(m->R + (size_t)row * H, hs, H);
        float x[3] = {orc_scale(cprev[st]), orc_scale(fprev[st]), 0.0f};
        /* coarse half, coarse head, coarse draw */
        gru_units(m, G, add, x, hs, hn, 0, Hh);
        head(m, m->O1, m->b1, m->O2, m->b2, hn, zc);
        float uc, uf;
        orc_uniforms(seed, (uint64_t)st, B == 1 ? n : i, &uc, &uf);
        int c = tgt ? (tgt[local] >> 8) : orc_draw(zc, ORC_MAX_CLASSES, uc);
        /* fine half sees c_t, fine head, fine draw */
        x[2] = orc_scale(c);
        gru_units(m, G, add, x, hs, hn, Hh, H);
        head(m, m->O3, m->b3, m->O4, m->b4, hn + Hh, zf);
        int f = tgt ? (tgt[local] & 255) : orc_draw(zf, ORC_MAX_CLASSES, uf);
        memcpy(hs, hn, sizeof(float) * H);
        cprev[st] = (uint8_t)c;
        fprev[st] = (uint8_t)f;
        if (!tgt) seq[local] = (uint16_t)(256 * c + f);
        else if (seq) seq[local] = tgt[local];
        size_t o = (size_t)s * T + local;
        if (zc_out) memcpy(zc_out + o * ORC_MAX_CLASSES, zc, sizeof zc);
        if (zf_out) memcpy(zf_out + o * ORC_MAX_CLASSES, zf, sizeof zf);
        if (nll_out) nll_out[o] = neg_log_prob(zc, ORC_MAX_CLASSES, c) + neg_log_prob(zf, ORC_MAX_CLASSES, f);
      }
    }
  }
  free(G); free(add); free(hn); free(ctx); free(ctab);
  return 0;
}

int orc_run(const orc_model* m, int32_t S, int64_t T, int64_t t0, const float* feat, int64_t n_frames,
            uint64_t seed, const uint16_t* target, float* h, uint8_t* cprev, uint8_t* fprev, uint16_t* out,
            float* zc_out, float* zf_out, double* nll_out) {
  return run_lanes(m, S, T, t0, feat, n_frames, seed, target, h, cprev, fprev, out, zc_out, zf_out, nll_out, 0,
                   m->B > 0 ? m->B : 1);
}

int orc_run_lanes(const orc_model* m, int32_t S, int64_t T, const float* feat, int64_t n_frames,
                  const uint16_t* target, float* h, uint8_t* cprev, uint8_t* fprev, float* zc_out, float* zf_out,
                  double* nll_out, int32_t lane_lo, int32_t lane_hi) {
  return run_lanes(m, S, T, 0, feat, n_frames, 0, target, h, cprev, fprev, NULL, zc_out, zf_out, nll_out, lane_lo,
                   lane_hi);
}

/* ------------------------------------------------------------------------- */
/* Fused Subscale WaveRNN 2x (Sec. 4.4)                                        */
/* ------------------------------------------------------------------------- */
/* The paper describes the model in a few sentences: a Subscale 2x model whose
 * two sub-tensors, instead of being batched, share one WaveRNN by splitting
 * its state, with 8 softmaxes of 4 bits and a future horizon of 2, the
 * samples entering the WaveRNN directly as inputs.  Readings fixed here:
 *   - units [0,Q) are the coarse quarter of sub-tensor 0, [Q,2Q) the coarse
 *     quarter of sub-tensor 1, [2Q,3Q) and [3Q,4Q) their fine quarters
 *     (Q = H/4); R is one full 3H x H matrix (the state is one vector);
 *   - step t runs position t of sub-tensor 0 and position t - (F + 1) of
 *     sub-tensor 1, so the state that makes position i of sub-tensor 1 has
 *     seen sub-tensor 0 up to position i + F (Sec. 4.2);
 *   - inputs x = (c0, f0, c1, f1) of each sub-tensor's last sample, then the
 *     coarse bytes c0_t, c1_t of this step: the coarse quarters use the first
 *     four columns of I, the fine quarter of sub-tensor s those four and the
 *     column of its own c_t (the I* mask of Eq. 2 per sub-tensor: the coarse
 *     half is evaluated and its bytes drawn before the fine half), so the two
 *     parts meet only through the state and the last samples;
 *   - each byte is two nibbles (high, low) drawn from two 16-way softmaxes of
 *     one output head per (level, sub-tensor), k = 2 level + s:
 *     o = relu(O1_k y + b1_k) on that quarter y, z_hi = O2_k,hi o + b2_k,hi,
 *     z_lo = O2_k,lo o + b2_k,lo, byte = 16 hi + lo; the two nibbles of a byte
 *     are independent given the state (8 softmaxes per step, 32 bits);
 *   - a sub-tensor outside its positions (sub-tensor 1 for the first F + 1
 *     steps, sub-tensor 0 for the last F + 1) is idle: it draws nothing and
 *     its inputs, its coarse-byte input included, keep its last sample
 *     (before the first: c = 128, f = 0);
 *   - conditioning: a unit of sub-tensor s adds W_cond times the frame of the
 *     sample its sub-tensor makes (its last position while idle);
 *   - uniforms: Philox4x64-10, key (seed, 0), counter (i, 2 u + s, 0, 0) for
 *     position i of sub-tensor s of utterance u; words 0..3 give the coarse
 *     high, coarse low, fine high and fine low nibble.
 * Sample n = 2 i + s of an utterance is position i of sub-tensor s. */

/* A (level, sub-tensor) head: z[0..15] high nibble, z[16..31] low nibble. */
static void fused_head(const orc_fused_model* m, int k, const float* y, float* z) {
  const int Q = m->H / 4;
  float hid[ORC_MAX_HIDDEN / 4];
  const float* Oa = m->O1 + (size_t)k * Q * Q;
  const float* ba = m->b1 + (size_t)k * Q;
  for (int j = 0; j < Q; ++j) hid[j] = relu(dot(Oa + (size_t)j * Q, y, Q) + ba[j]);
  for (int v = 0; v < 32; ++v)
    z[v] = dot(m->O2 + ((size_t)k * 32 + v) * Q, hid, Q) + m->b2[(size_t)k * 32 + v];
}

/* Gates of units [lo, hi) with the first nx input columns (of six). */
static void fused_units(const orc_fused_model* m, const float* G, const float* add, const float* x, int nx,
                        const float* h_prev, float* h_new, int lo, int hi) {
  const int H = m->H;
  for (int i = lo; i < hi; ++i) {
    float ix[3];
    for (int g = 0; g < 3; ++g) ix[g] = dot(m->I + ((size_t)g * H + i) * 6, x, nx);
    const float ug = orc_sigmoid(G[0 * H + i] + (ix[0] + add[0 * H + i]));
    const float rg = orc_sigmoid(G[1 * H + i] + (ix[1] + add[1 * H + i]));
    const float eg = orc_tanh(fmaf(rg, G[2 * H + i], ix[2] + add[2 * H + i]));
    h_new[i] = fmaf(ug, h_prev[i], (1.0f - ug) * eg);
  }
}

static int fused_nibbles(const float* z, const float* u, int forced) {
  if (forced >= 0) return forced;
  return 16 * orc_draw(z, 16, u[0]) + orc_draw(z + 16, 16, u[1]);
}

int orc_fused_run(const orc_fused_model* m, int32_t S, int64_t N, const float* feat, int64_t n_frames,
                  uint64_t seed, const uint16_t* target, uint16_t* out, float* zc_out, float* zf_out,
                  double* nll_out, float* h_final) {
  const int H = m->H, Q = H / 4;
  if (H <= 0 || H % 4 || H > ORC_MAX_HIDDEN || S <= 0 || N < 0 || N % 2 || m->F < 0) return -1;
  if (m->Dc > 0 && (m->frame_len <= 0 || feat == NULL || n_frames <= 0)) return -1;
  if (target == NULL && out == NULL) return -1;
  const int64_t rows = N / 2, steps = N > 0 ? rows + m->F + 1 : 0;
  float* h = (float*)malloc(sizeof(float) * H);
  float* hn = (float*)malloc(sizeof(float) * H);
  float* G = (float*)malloc(sizeof(float) * 3 * H);
  float* add = (float*)malloc(sizeof(float) * 3 * H);
  for (int32_t ut = 0; ut < S; ++ut) {
    const uint16_t* tgt = target ? target + (size_t)ut * N : NULL;
    for (int i = 0; i < H; ++i) h[i] = 0.0f;
    int cl[2] = {128, 128}, fl[2] = {0, 0};            /* last sample of each sub-tensor */
    for (int64_t t = 0; t < steps; ++t) {
      const int64_t p[2] = {t, t - (m->F + 1)};
      const int act[2] = {p[0] >= 0 && p[0] < rows, p[1] >= 0 && p[1] < rows};
      int64_t nn[2];                                   /* the sample each sub-tensor makes (or made last) */
      for (int s = 0; s < 2; ++s) {
        int64_t pc = p[s] < 0 ? 0 : (p[s] >= rows ? rows - 1 : p[s]);
        nn[s] = 2 * pc + s;
      }
      for (int row = 0; row < 3 * H; ++row) {
        const int s = (row % H) / Q % 2;
        float bias_cond = m->b[row];
        if (m->Dc > 0) {
          int64_t fr = nn[s] / m->frame_len;
          if (fr >= n_frames) fr = n_frames - 1;
          bias_cond = dot(m->Wc + (size_t)row * m->Dc, feat + ((size_t)ut * n_frames + fr) * m->Dc, m->Dc) + m->b[row];
        }
        add[row] = bias_cond;
        G[row] = dot(m->R + (size_t)row * H, h, H);
      }
      float u[2][4];
      for (int s = 0; s < 2; ++s) {
        uint64_t ctr[4] = {(uint64_t)(act[s] ? p[s] : 0), (uint64_t)(2 * ut + s), 0, 0}, key[2] = {seed, 0}, w[4];
        orc_philox4x64_10(ctr, key, w);
        for (int k = 0; k < 4; ++k) u[s][k] = (float)(w[k] >> 40) * (1.0f / 16777216.0f);
      }
      float x[6] = {orc_scale(cl[0]), orc_scale(fl[0]), orc_scale(cl[1]), orc_scale(fl[1]), 0.0f, 0.0f};
      float zc[2][32], zf[2][32];
      int c[2], f[2];
      /* coarse half, the two coarse heads, the coarse bytes */
      fused_units(m, G, add, x, 4, h, hn, 0, 2 * Q);
      for (int s = 0; s < 2; ++s) {
        fused_head(m, s, hn + s * Q, zc[s]);
        c[s] = act[s] ? fused_nibbles(zc[s], u[s], tgt ? tgt[2 * p[s] + s] >> 8 : -1) : cl[s];
      }
      /* each fine quarter sees its own coarse byte; the two fine heads, the fine bytes */
      x[4] = orc_scale(c[0]);
      fused_units(m, G, add, x, 6, h, hn, 2 * Q, 3 * Q);
      x[4] = 0.0f;
      x[5] = orc_scale(c[1]);
      fused_units(m, G, add, x, 6, h, hn, 3 * Q, 4 * Q);
      for (int s = 0; s < 2; ++s) {
        fused_head(m, 2 + s, hn + 2 * Q + s * Q, zf[s]);
        f[s] = act[s] ? fused_nibbles(zf[s], u[s] + 2, tgt ? tgt[2 * p[s] + s] & 255 : -1) : fl[s];
      }
      memcpy(h, hn, sizeof(float) * H);
      for (int s = 0; s < 2; ++s) {
        if (!act[s]) continue;
        const size_t o = (size_t)ut * N + (size_t)(2 * p[s] + s);
        if (out) out[o] = (uint16_t)(256 * c[s] + f[s]);
        if (zc_out) memcpy(zc_out + o * 32, zc[s], sizeof zc[s]);
        if (zf_out) memcpy(zf_out + o * 32, zf[s], sizeof zf[s]);
        if (nll_out)
          nll_out[o] = neg_log_prob(zc[s], 16, c[s] >> 4) + neg_log_prob(zc[s] + 16, 16, c[s] & 15) +
                       neg_log_prob(zf[s], 16, f[s] >> 4) + neg_log_prob(zf[s] + 16, 16, f[s] & 15);
        cl[s] = c[s];
        fl[s] = f[s];
      }
    }
    if (h_final) memcpy(h_final + (size_t)ut * H, h, sizeof(float) * H);
  }
  free(h); free(hn); free(G); free(add);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Subscale conditioning network: masked dilated 1-D CNN (Sec. 4.1, 5)         */
/* ------------------------------------------------------------------------- */
/* The paper: a masked dilated CNN with relus whose mask is applied over past
 * connections instead of future ones, conditioning each sub-tensor on the
 * past and future of the previous sub-tensors; ten layers, kernel size 3,
 * 384 convolution channels, 768 residual channels, 5 stages of increasing
 * dilation, a future horizon of 128 blocks of B samples.  Readings fixed here:
 *   - the network runs over rows (blocks) k of an utterance; the input of row
 *     k for sub-tensor s is the (c, f) pair, scaled, of every sub-tensor z of
 *     that row, zero for z >= s (the previous sub-tensors only) and zero for
 *     rows outside the utterance: 2B channels;
 *   - a 1x1 input layer maps them to Rc residual channels: r = Win x + bin;
 *   - layer l (dilation d = 2^(l mod 5)) reads r at rows k, k + d, k + 2d
 *     (the future taps: the mask removes the past ones), a = relu(sum over taps
 *     of Wc_l,tap r + bc_l) with Cc convolution channels, and adds Wo_l a + bo_l
 *     back into r (residual);
 *   - a 1x1 output layer gives the Dx-dim conditioning vector of row k:
 *     out = Wp r + bp.  Ten layers of dilations 1..16 see rows k .. k + 124.
 * The sub-tensor s at position i is conditioned on out(s, i), so it sees the
 * previous sub-tensors at rows i .. i + 124 directly and earlier rows through
 * its state (the unbounded past horizon). */
int orc_ctx_cnn(const orc_cnn* m, const uint16_t* seq, int64_t N, int32_t s, float* out) {
  const int B = m->B, Rc = m->Rc, Cc = m->Cc, Dx = m->Dx;
  if (B < 1 || N % B || s < 0 || s >= B || Rc <= 0 || Cc <= 0 || Dx <= 0 || m->layers < 0) return -1;
  const int64_t rows = N / B;
  float* r = (float*)malloc(sizeof(float) * (size_t)(rows > 0 ? rows : 1) * Rc);
  float* rn = (float*)malloc(sizeof(float) * (size_t)(rows > 0 ? rows : 1) * Rc);
  float* x = (float*)malloc(sizeof(float) * 2 * B);
  float* a = (float*)malloc(sizeof(float) * Cc);
  for (int64_t k = 0; k < rows; ++k) {
    for (int z = 0; z < B; ++z) {
      const int seen = z < s;
      x[2 * z] = seen ? orc_scale(seq[B * k + z] >> 8) : 0.0f;
      x[2 * z + 1] = seen ? orc_scale(seq[B * k + z] & 255) : 0.0f;
    }
    for (int o = 0; o < Rc; ++o) r[k * Rc + o] = dot(m->Win + (size_t)o * 2 * B, x, 2 * B) + m->bin[o];
  }
  for (int l = 0; l < m->layers; ++l) {
    const int d = 1 << (l % 5);
    const float* Wc = m->Wc + (size_t)l * Cc * 3 * Rc;   /* [Cc][3][Rc] */
    const float* Wo = m->Wo + (size_t)l * Rc * Cc;       /* [Rc][Cc] */
    for (int64_t k = 0; k < rows; ++k) {
      for (int c = 0; c < Cc; ++c) {
        float acc = m->bc[(size_t)l * Cc + c];
        for (int tap = 0; tap < 3; ++tap) {
          const int64_t kk = k + (int64_t)tap * d;      /* future taps only */
          if (kk >= rows) continue;                      /* beyond the utterance: zero */
          acc = acc + dot(Wc + ((size_t)c * 3 + tap) * Rc, r + kk * Rc, Rc);
        }
        a[c] = relu(acc);
      }
      for (int o = 0; o < Rc; ++o)
        rn[k * Rc + o] = r[k * Rc + o] + (dot(Wo + (size_t)o * Cc, a, Cc) + m->bo[(size_t)l * Rc + o]);
    }
    memcpy(r, rn, sizeof(float) * (size_t)rows * Rc);
  }
  for (int64_t k = 0; k < rows; ++k)
    for (int o = 0; o < Dx; ++o) out[k * Dx + o] = dot(m->Wp + (size_t)o * Rc, r + k * Rc, Rc) + m->bp[o];
  free(r); free(rn); free(x); free(a);
  return 0;
}
