/*
 * wavernn.h -- C ABI of libwavernn, WaveRNN sampling on MI355X (gfx950).
 *
 * The library implements the sampling step of "Efficient Neural Audio
 * Synthesis" (Kalchbrenner et al., 2018): the single GRU layer of Eq. 2 with
 * the masked input matrix I* (Sec. 2, text after Eq. 2), the dual 8-bit softmax
 * (coarse byte first, then the fine byte conditioned on it; Fig. 1 caption),
 * draws from the two softmaxes, repeated once per 16-bit audio sample, as one
 * persistent GPU operation per call (Sec. 2.1).  It also covers block-sparse R
 * (Sparse WaveRNN, Sec. 3.2: 4x4 and 16x1 blocks) and subscale batching
 * (Subscale WaveRNN, Sec. 4, Eq. 4).
 *
 * Conventions shared by every entry point:
 *  - Weights are passed as host fp32 arrays, row-major, gate order u, r, e.
 *    The library copies them (the caller may free them on return), applies the
 *    I* mask, rounds to bf16 (round to nearest even) if asked, packs them for
 *    the kernels and owns the device copies until wavernn_destroy.
 *  - Every other buffer is caller-owned *device* memory.  Calls are
 *    asynchronous and ordered on the given HIP stream (hipStream_t passed as
 *    void*, NULL = the null stream); inputs must stay valid until the work on
 *    that stream is done.
 *  - A 16-bit sample is stored offset-binary: u = 256*c + f, c the coarse
 *    (high) byte, f the fine (low) byte (Fig. 1 caption).  Bytes enter the
 *    network scaled to [-1, 1] as (2v - 255) / 255 (Sec. 2).
 *  - Draws use Philox4x64-10 (Salmon et al., SC'11), key (seed, 0), counter
 *    (t, stream, 0, 0) with t the absolute step; word 0 gives the coarse
 *    uniform, word 1 the fine one, U = (word >> 40) * 2^-24.  A class is
 *    drawn by inverse CDF over exp(z - max z).
 *  - Functions return a wavernn_status; on failure nothing is launched and
 *    wavernn_last_error() (per thread) describes the cause.  No exceptions
 *    cross the ABI.
 *  - A model serves one call at a time.  Every sample, score and sync-floor
 *    call of a model uses the model's own exchange words, per-frame tables and
 *    error word, so two calls of one model whose GPU work overlaps (on two
 *    streams, or from two threads) race and may time out or corrupt each
 *    other; calls queued on one stream are safe.  Separate models are
 *    independent.
 *  - A failure a kernel flags (a bounded wait that expired) stays recorded in
 *    the model's error word: the launch that flagged it ends early, and every
 *    later launch of the model ends at the first wait that has to spin (the
 *    outputs of those launches are undefined) while the launching calls still
 *    return WAVERNN_OK, until wavernn_device_status reports WAVERNN_E_DEVICE
 *    and clears the word.  Check wavernn_device_status after work whose
 *    outputs matter.
 */
#ifndef WAVERNN_H
#define WAVERNN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WAVERNN_OK = 0,
  WAVERNN_E_INVALID = 1,      /* bad argument: null pointer, shape, size, range */
  WAVERNN_E_UNSUPPORTED = 2,  /* valid request the library cannot run (e.g. grid cannot be co-resident) */
  WAVERNN_E_OOM = 3,          /* device allocation failed */
  WAVERNN_E_HIP = 4,          /* a HIP runtime call failed */
  WAVERNN_E_DEVICE = 5        /* the kernel reported a failure (wavernn_device_status) */
} wavernn_status;

typedef enum { WAVERNN_F32 = 0, WAVERNN_BF16 = 1 } wavernn_dtype;

/* Storage of R.  BSR formats keep the blocks the mask marks (Sec. 3.2):
 * 4x4 blocks, or 16x1 blocks (16 consecutive rows of one column). */
typedef enum { WAVERNN_R_DENSE = 0, WAVERNN_R_BSR_4X4 = 1, WAVERNN_R_BSR_16X1 = 2 } wavernn_r_format;

typedef struct {
  int32_t hidden;        /* H: hidden units, even; H/2 coarse, H/2 fine (Eq. 2 split) */
  int32_t cond_dim;      /* Dc: conditioning features per frame, 0 = none */
  int32_t frame_len;     /* samples per conditioning frame (> 0 when cond_dim > 0) */
  int32_t subscale;      /* B: samples per step per utterance, 1 (plain) or > 1 (Sec. 4) */
  int32_t ctx_dim;       /* Dx: subscale context width (2 per context sample), 0 when B = 1 */
  int32_t weight_dtype;  /* wavernn_dtype of the stored weights; arithmetic is fp32 */
  int32_t r_format;      /* wavernn_r_format */
  int32_t max_streams;   /* most utterances one call may sample, 1..64 */
  int32_t future_horizon; /* F, subscale only (ignored when B = 1): -1 = lockstep rows (all B lanes
                            make row i together, each seeing the Dx/2 samples before its own of
                            earlier rows); F >= 0 = the paper's order with future horizon F
                            (Sec. 4.2): sample B*i + s sees sub-tensors z < s up to position i + F
                            (its own sub-tensor through the state only), its context the Dx/4 samples before
                            and Dx/4 after it (unseen ones zero); lane s runs position i at step
                            i + s(F + 1 + A), so a call takes n_samples/B + (B - 1)(F + 1 + A)
                            steps.  0 is a valid horizon: set -1 for lockstep. */
  int32_t context_lead;   /* A in [0, 3], only with a future horizon (must be 0 otherwise; ignored
                            when B = 1): each sub-tensor starts A steps later than the horizon
                            alone requires, so that the samples its context needs were drawn A
                            steps before the step that uses them and the context is formed off
                            the step's critical chain (Sec. 4.2: the conditioning runs ahead of
                            the lane it feeds).  The samples drawn do not depend on A.
                            Currently switched off: create returns E_UNSUPPORTED for A > 0. */
  int32_t fused;          /* 1 = Fused Subscale WaveRNN 2x (Sec. 4.4): the two sub-tensors of a
                            Subscale 2x model share one WaveRNN by splitting its state into
                            quarters (units [0, H/4) coarse of sub-tensor 0, [H/4, H/2) coarse of
                            sub-tensor 1, then their fine quarters), each byte is drawn as two
                            4-bit nibbles from 16-way softmaxes (8 per step), and sub-tensor 1
                            runs future_horizon + 1 steps behind sub-tensor 0 (the paper uses 2).
                            Needs subscale = 2, ctx_dim = 0, context_lead = 0, future_horizon
                            >= 0, dense bf16 R and an H the batch-1 kernel serves (a multiple of
                            128 up to 896).  Sample 2 i + s of an utterance is position i of
                            sub-tensor s; a call takes n_samples / 2 + F + 1 steps.  0 = plain. */
} wavernn_config;

/* Host fp32 weights.  Shapes (H hidden, Hh = H/2, V = 256 classes):
 *   R [3][H][H], R_block_mask [3][H/bh][H/bw] (uint8, nonzero = kept; only for BSR),
 *   I [3][H][3] columns (c_{t-1}, f_{t-1}, c_t): column 2 of rows i < Hh is ignored (I* mask),
 *   b [3][H], W_cond [3H][Dc], W_ctx [3H][Dx],
 *   O1 [Hh][Hh], b1 [Hh], O2 [V][Hh], b2 [V] (coarse head, Eq. 2),
 *   O3 [Hh][Hh], b3 [Hh], O4 [V][Hh], b4 [V] (fine head).
 * For BSR formats, entries of R outside kept blocks are ignored.
 * Fused 2x models (Q = H/4) take instead:
 *   I [3][H][6] columns (c0, f0, c1, f1) of each sub-tensor's last sample, then
 *     c0_t, c1_t of this step; the coarse half reads columns 0-3 only, the fine
 *     quarter of sub-tensor s columns 0-3 and 4 + s (the others are ignored);
 *   O1 [4][Q][Q], b1 [4][Q]: first layer of head k = 2 level + s (level 0 coarse,
 *     1 fine) on quarter k of the state; O2 [4][2][16][Q], b2 [4][2][16]: its
 *     high-nibble and low-nibble logits; O3, b3, O4, b4 are unused (may be NULL). */
/* The masked dilated 1-D CNN that conditions a Subscale WaveRNN on the
 * previous sub-tensors (Sec. 4.1; shape in Sec. 5: ten layers, kernel size 3,
 * 384 convolution channels, 768 residual channels, five stages of increasing
 * dilation).  It runs over rows k (blocks of B samples).  The input of row k
 * for sub-tensor s is the (c, f) pair, scaled as every byte, of each
 * sub-tensor z < s of that row (2B channels, zero for z >= s and outside the
 * utterance):  r = Win x + bin;  then for each layer l (dilation
 * d = 2^(l mod 5)), with the mask keeping the future taps only,
 *   a = relu(Wc_l [r_k ; r_k+d ; r_k+2d] + bc_l)  (rows past the end: zero),
 *   r = r + (Wo_l a + bo_l);
 * and the context vector of row k is Wp r + bp (Dx = the model's ctx_dim).
 * Ten layers see rows k .. k + 124.  Sub-tensor s at position i is
 * conditioned on its vector of row i, through W_ctx as the window context is.
 * Res/conv channels and Dx must be multiples of 128; weights are rounded to
 * bf16 like the model's. */
typedef struct {
  int32_t res_channels;    /* Rc */
  int32_t conv_channels;   /* Cc */
  int32_t layers;          /* >= 0 */
  const float *Win, *bin;  /* [Rc][2B], [Rc] */
  const float *Wc, *bc;    /* [layers][Cc][3][Rc] (taps k, k + d, k + 2d), [layers][Cc] */
  const float *Wo, *bo;    /* [layers][Rc][Cc], [layers][Rc] */
  const float *Wp, *bp;    /* [Dx][Rc], [Dx] */
} wavernn_ctx_cnn;

typedef struct {
  const float* R;
  const uint8_t* R_block_mask;
  const float* I;
  const float* b;
  const float* W_cond;
  const float* W_ctx;
  const float *O1, *b1, *O2, *b2, *O3, *b3, *O4, *b4;
  const wavernn_ctx_cnn* ctx_cnn;   /* subscale with a future horizon only: the conditioning CNN that
                                       replaces the window context; NULL = window context */
} wavernn_weights;

/* Recurrent state of S utterances x B lanes, device memory:
 * h [S*B][H] fp32, c_prev / f_prev [S*B] bytes of the previous sample,
 * t0 = absolute index of the next sample (B = 1 only; 0 otherwise).
 * Fused 2x models: h [S][H] (one state per utterance), c_prev / f_prev [2S]
 * the last sample of sub-tensors 0 and 1 of each utterance, t0 = 0.
 * Default initial state: h = 0, c_prev = 128, f_prev = 0, t0 = 0. */
typedef struct {
  float* h;
  uint8_t* c_prev;
  uint8_t* f_prev;
  int64_t t0;
} wavernn_state;

typedef struct wavernn_model wavernn_model;

/* Validate cfg, copy and pack the weights to the current HIP device.
 * *out receives the model handle.  Errors: E_INVALID (null pointer, odd or
 * unsupported H, bad config field), E_UNSUPPORTED (no kernel of the library
 * serves the configuration), E_OOM, E_HIP. */
wavernn_status wavernn_create(const wavernn_config* cfg, const wavernn_weights* w, wavernn_model** out);

/* Free the model's device memory.  Null-safe.  Work already queued that uses
 * the model must have finished. */
void wavernn_destroy(wavernn_model* m);

/* Sample n_samples 16-bit samples for each of n_streams utterances (Eq. 2,
 * dual softmax, Fig. 1 order), as one persistent kernel launch per call.
 *   cond_dev  [n_streams][n_frames][Dc] fp32 feature frames; frame index of
 *             absolute sample n is n / frame_len (NULL when Dc = 0)
 *   init      initial state (NULL = default); out_dev [n_streams][n_samples] uint16
 *   final     where to write the state after the last sample (NULL = nowhere);
 *             may alias init.
 * Subscale (B > 1): n_samples must be a multiple of B; lane s of step i makes
 * sample B*i + s and out_dev is in time order.  Utterance k draws from Philox
 * stream k*B + lane.  n_samples = 0 is valid: nothing is launched and final
 * is left as it was.  Errors: E_INVALID, E_UNSUPPORTED, E_HIP. */
wavernn_status wavernn_sample(wavernn_model* m, int32_t n_streams, int64_t n_samples, const float* cond_dev,
                              int64_t n_frames, uint64_t seed, const wavernn_state* init, uint16_t* out_dev,
                              const wavernn_state* final_state, void* stream);

/* Subscale models on the batched path (B > 1, not fused; Sec. 4): run steps
 * [step0, step0 + n_steps) of the schedule of a call of n_samples samples per
 * utterance, so that an utterance can be generated over several calls
 * (streaming, or resuming from a saved state).  The schedule has
 * wavernn_schedule_steps(m, n_samples) steps; step i runs position
 * i - s (F + 1) of lane s with a future horizon F (Sec. 4.2), position i of
 * every lane without one, and lane s at position p makes sample B p + s.
 *   out_dev   [n_streams][n_samples] uint16: the whole utterances.  The call
 *             writes the samples its steps make and reads, for the context of
 *             its first steps, the ones earlier steps made, which earlier calls
 *             must have written there.
 *   init      the state after step step0 - 1 (required when step0 > 0; NULL =
 *             default when step0 = 0); final: the state after the call's last
 *             step (NULL = nowhere; may alias init).  Both with t0 = 0.
 *   cond_dev, n_frames, seed: as for one wavernn_sample call of n_samples.
 * Running steps [0, K) in any number of calls makes the same samples and
 * final state as one wavernn_sample call, bit for bit.  The samples of lane s
 * up to position p are final once step p + s (F + 1) has run.  n_steps = 0
 * is valid (nothing launched).  Errors: E_INVALID (step range, missing init,
 * as wavernn_sample), E_UNSUPPORTED (not a subscale model on the batched path;
 * step0 > 0 with the window context and B not a power of two), E_HIP. */
wavernn_status wavernn_sample_steps(wavernn_model* m, int32_t n_streams, int64_t n_samples, const float* cond_dev,
                                    int64_t n_frames, uint64_t seed, int64_t step0, int64_t n_steps,
                                    const wavernn_state* init, uint16_t* out_dev, const wavernn_state* final_state,
                                    void* stream);
/* Steps of the schedule of a subscale call of n_samples samples per utterance
 * (n_samples / B, plus (B - 1)(F + 1) with a future horizon F); -1 for a model
 * that wavernn_sample_steps does not serve or an invalid n_samples. */
int64_t wavernn_schedule_steps(const wavernn_model* m, int64_t n_samples);

/* wavernn_sample without any device allocation, for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, kernels and results as wavernn_sample
 * (bit for bit), but the exchange words and the per-frame bias + conditioning
 * tables of the call live in a workspace the library holds per device: a
 * static device array of 16 MiB, kept until the process
 * ends, never in buffers the model grows.  A call needs, per launch, the
 * exchange words (under 64 KiB) plus n_frames * 3 * hidden * 4 bytes of table
 * (per utterance on the batched path; 2-4 concurrent utterances take one
 * launch each), each part rounded up to 256 bytes; a call that needs more
 * than 16 MiB fails with E_INVALID before anything is launched (WaveRNN-896
 * with 64-dim frames of 120 samples: up to about 1,500 frames, 7.5 s, per
 * utterance at batch 1).  The workspace is shared by every model and call on
 * the device and keeps the last call's contents (each call clears what must
 * start at zero and writes every table entry it reads): no-allocation calls
 * whose GPU work overlaps on one device race, whichever model they use.
 * Errors: as wavernn_sample, E_HIP if the workspace's address cannot be
 * looked up. */
wavernn_status wavernn_sample_noalloc(wavernn_model* m, int32_t n_streams, int64_t n_samples, const float* cond_dev,
                                      int64_t n_frames, uint64_t seed, const wavernn_state* init, uint16_t* out_dev,
                                      const wavernn_state* final_state, void* stream);

/* Teacher-forced scoring of known audio (the NLL of Sec. 5): the recurrence
 * runs on target_dev [n_streams][n_samples] instead of drawn samples.  Writes
 * the pre-softmax logits logits_c_dev / logits_f_dev [n_streams][n_samples][256]
 * and nll_dev [n_streams][n_samples] = -log P(c_t) - log P(f_t | c_t) in nats;
 * each output pointer may be NULL.  Fused 2x models write 32 logits per
 * sample and byte instead of 256 (high nibble 16, then low nibble 16), and
 * the NLL is the sum over the sample's four nibbles.  Initial state as in wavernn_sample.
 * n_samples = 0 is valid (target_dev may then be NULL): nothing is launched.
 * One utterance of a dense model on the multi-workgroup persistent path
 * (or several, one after another, on a model made for one) scores on a
 * recurrence-only kernel (with the bytes given, a step only updates h: one
 * exchange per step) and then runs the output layers over all steps as
 * matrix-core GEMMs.  That path keeps h of every step (4 H bytes per sample)
 * and the output layers' intermediates (4 (Hh rounded up to 128) + 2 KiB per
 * sample, for at most 65,536 samples at a time) in model-owned buffers, grown
 * the first time a longer call needs them; its initial state, conditioning
 * and outputs are as above. */
wavernn_status wavernn_score_teacher_forced(wavernn_model* m, int32_t n_streams, int64_t n_samples,
                                            const float* cond_dev, int64_t n_frames, const uint16_t* target_dev,
                                            const wavernn_state* init, float* logits_c_dev, float* logits_f_dev,
                                            float* nll_dev, void* stream);

/* Wait for the model's last call on `stream` and report a failure the kernel
 * flagged (a bounded wait that expired): WAVERNN_OK or WAVERNN_E_DEVICE. */
wavernn_status wavernn_device_status(wavernn_model* m, void* stream);

/* Philox uniforms as the device computes them: out_dev [n][2] fp32 =
 * (coarse, fine) uniforms of steps t0 .. t0+n-1 on `stream_id`. */
wavernn_status wavernn_debug_uniforms(uint64_t seed, uint64_t stream_id, int64_t t0, int64_t n, float* out_dev,
                                      void* stream);

/* Which kernel serves a call on n_streams streams: 0 single-workgroup fp32,
 * 1 multi-workgroup persistent (one launch per stream, one after another),
 * 2 batched persistent (up to 64 streams in one launch, 2, 4 or 8 per group
 * of workgroups; models created with max_streams > 1 and a hidden size the
 * persistent kernel serves, and every subscale model), 3 persistent with
 * block-sparse R (Sec. 3.2; one launch per stream), 4 concurrent persistent
 * (2 to 4 streams of a dense model whose grids fit the device together: one
 * batch-1 launch per stream on internal streams forked from and joined back
 * into the caller's stream; bit-identical to path 1), 5 fused 2x persistent
 * (Sec. 4.4; one launch per stream).
 * Fills *grid and *block with the launch shape of one launch; -1 for a null
 * model. */
int32_t wavernn_model_path(const wavernn_model* m, int32_t n_streams, int32_t* grid, int32_t* block);

/* Placement of the workgroups of the multi-workgroup persistent kernels
 * (paths 1, 3 and 5 of wavernn_model_path) among the 8 XCDs of the device.
 * Workgroups exchange values every step through memory, and the latency of
 * an exchange depends on where producer and consumer sit, in ways that
 * differ from device to device.  Candidate i (0 <= i < 64) puts the head
 * workgroups on XCD hx = i / 8 and the unit workgroups on XCD ux = i % 8
 * (ux == hx: the units spread over every XCD, the default, candidate 0).
 * A candidate fits when every workgroup of one launch can be resident at
 * once; only launches that run one at a time use the placement (the
 * concurrent launches of path 4 keep the default).  Results do not depend
 * on the placement: only the time per step does.
 *
 * wavernn_tune: times `rounds` (1..16) rounds of one sampling launch of
 * n_steps (16 .. 2^20) steps, zero conditioning, for each fitting candidate
 * on `stream`, and keeps the fastest for later calls.  us_out [64] (host
 * memory, or NULL) receives each candidate's best microseconds per step (-1
 * where it does not fit), *chosen (or NULL) the candidate kept.  Waits for
 * the stream; allocates and frees a few small device buffers; uses the
 * model's exchange buffer (no other call on the model may overlap it).  A
 * model on another path is left as it is (*chosen = -1).  Errors:
 * E_INVALID, E_HIP, E_DEVICE (a bounded wait expired in a launch of the
 * default placement). */
wavernn_status wavernn_tune(wavernn_model* m, int64_t n_steps, int32_t rounds, float* us_out, int32_t* chosen,
                            void* stream);
/* Sets the placement to candidate i (as in wavernn_tune), -1 for the
 * default.  E_INVALID if i is out of range or the candidate does not fit,
 * E_UNSUPPORTED for a model on another path. */
wavernn_status wavernn_set_placement(wavernn_model* m, int32_t candidate);

/* Diagnostics: make later wavernn_sample / wavernn_score_teacher_forced calls
 * of the multi-workgroup persistent kernel record, for the first max_steps
 * steps of the first utterance, timestamps of the 100 MHz constant clock at
 * the end of each phase of a step into trace_dev [max_steps][32] (device
 * memory the caller owns and keeps alive while tracing is on).  Slot 0 is
 * the start of the step on head workgroup 0; the other slots are the ends of
 * the phases of that step (gates, hidden layers, partial logits published,
 * logits summed, draws) on head workgroup 0 or on the last head workgroup;
 * unused slots stay zero.  max_steps = 0 turns tracing off.  Other kernels
 * ignore the setting.  A sampling or scoring call of a model with a
 * conditioning CNN returns E_UNSUPPORTED while tracing is on (switched off:
 * one traced call of that path had a bounded wait expire, cause not found). */
wavernn_status wavernn_set_trace(wavernn_model* m, uint64_t* trace_dev, int64_t max_steps);

/* Diagnostics: the synchronization floor of the model's persistent kernel
 * (paths 1 and 3 of wavernn_model_path).  Runs n_steps (>= 2) steps of a
 * kernel with the same grid, workgroup roles and exchanged words per step as
 * the sampling kernel but no arithmetic (the per-step synchronization cost
 * the paper discusses in Sec. 2.1), waits for it on `stream`, and writes its
 * mean time per step in microseconds to *us_per_step (host memory).  Uses the
 * model's exchange buffer: calls on other streams must not overlap it.
 * Errors: E_INVALID (arguments), E_UNSUPPORTED (other paths), E_HIP,
 * E_DEVICE (a bounded wait expired). */
wavernn_status wavernn_debug_sync_floor(wavernn_model* m, int64_t n_steps, double* us_per_step, void* stream);

/* The conditioning CNN of a model created with ctx_cnn (Sec. 4.1) over whole
 * utterances: out_dev [n_streams][B][n_samples / B][Dx] fp32 receives the
 * context vector of every sub-tensor s and row k from the samples seq_dev
 * [n_streams][n_samples] (n_samples a multiple of B).  Every layer runs as one
 * matrix-core GEMM over all rows of all sub-tensors, activations at fp32
 * accuracy (bf16 high and low parts) against the bf16 weights.  Scratch
 * activations are the model's (grown on demand: 4 (Rc + Cc + 32) bytes per
 * row of every sub-tensor).  Errors: E_INVALID (no CNN, bad sizes), E_OOM,
 * E_HIP. */
wavernn_status wavernn_ctx_cnn_run(wavernn_model* m, int32_t n_streams, int64_t n_samples, const uint16_t* seq_dev,
                                   float* out_dev, void* stream);

/* Description of the last error on this thread ("" if none). */
const char* wavernn_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
