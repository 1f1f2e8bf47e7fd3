// Batched persistent WaveRNN sampler: up to 64 independent utterances, or
// the lanes of subscale rows, per launch in groups of L = 2, 4 or 8 vectors
// (Sec. 2.1: many utterances share one GPU; Sec. 4: B samples per step).
//
// A group is the batch-1 structure of wr_persist.hip serving L vectors at
// once.  Every matrix-vector product of the step becomes an L-row product on
// the matrix cores at the same instruction count: operand A holds vector b in
// rows 2b (bf16 high part) and 2b+1 (remainder), and lane l of the result
// holds vectors 2(l/16) and 2(l/16)+1 of row l%16.  Per step and half the
// heads run their O1 rows / O2 columns for all vectors and publish L x 256
// partial logits.  With L <= 4 every head evaluates every gate of every
// vector and sums and draws every vector; with L = 8 head j evaluates the
// gates of its own 64 units for all vectors and the heads exchange those
// slices of y, and vector v is owned by head v mod NH, which alone sums its
// partials, draws it and publishes its classes.
#include "wr_kern.h"

namespace {


// Vector v is lane s = v % B of utterance v / B.  At step t it runs position
// p = vpos(v, t) and makes sample n = B (t0 + p) + s of that utterance
// (Sec. 4; B = 1: n = t0 + t): p = t for lockstep rows; with future horizon F
// (Sec. 4.2: a sub-tensor starts F + 1 steps after the one before it, A more
// when its context is formed A steps ahead, so the lanes of one step are at
// different positions and a lane idles before its first and after its last
// position) t0 is the schedule step the launch starts at, p = t0 + t -
// s (F + 1 + A) is the lane's absolute position and n = B p + s.
// (LAG: the kernel instantiated for a horizon schedule; lockstep kernels pay nothing for it.)
template <bool LAG>
__device__ __forceinline__ int64_t vpos(const BatchArgs& a, int v, int64_t t) {
  if (!LAG) return t;
  return a.t0 + t - (int64_t)(v % a.B) * (a.F + 1 + a.A);
}
// Index of sample B p + s in the [U][B rows] output / target arrays: obase(v) + B p.
__device__ __forceinline__ size_t obase(const BatchArgs& a, int v) {
  return (size_t)(v / a.B) * a.B * a.rows + v % a.B;
}
// Offset (floats) of the bias + conditioning row vector v uses at step t
// (an idle lane's position clamped to its first or last).
template <bool LAG>
__device__ __forceinline__ int64_t cb_offset(const BatchArgs& a, int v, int64_t t) {
  int64_t p = vpos<LAG>(a, v, t);
  if (LAG) p = p < 0 ? 0 : p >= a.rows ? a.rows - 1 : p;
  int64_t fr = ((int64_t)a.B * ((LAG ? 0 : a.t0) + p) + v % a.B) / a.frame_len;
  if (fr >= a.n_cb) fr = a.n_cb - 1;
  return ((int64_t)(v / a.B) * a.n_cb + fr) * 3 * a.P.H;
}

// Wait until the N words base[k*stride] (k < N) carry `tag`; values to v[].
template <int N>
__device__ __forceinline__ bool poll_strided(const xw* base, int stride, uint32_t tag, float* v, const BatchArgs& a) {
  uint64_t pending = N >= 64 ? ~0ull : (1ull << N) - 1ull;
  WaitBudget wb{wr_clock(), 0};
  for (;;) {
    xw w[N];
#pragma unroll
    for (int k = 0; k < N; ++k) w[k] = (pending >> k & 1ull) ? xpeek(base + (size_t)k * stride) : 0;
#pragma unroll
    for (int k = 0; k < N; ++k)
      if ((pending >> k & 1ull) && xok(w[k], tag)) {
        v[k] = xval(w[k]);
        pending &= ~(1ull << k);
      }
    if (!pending) return true;
    if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
}

// A pointer the compiler must treat as recomputed here: keeps address
// arithmetic inside the step loop instead of hoisting dozens of 64-bit
// addresses into registers for the whole launch.
template <class T>
__device__ __forceinline__ T* opaque(T* p) {
  asm volatile("" : "+v"(p));
  return p;
}

// Delay (x 64 clocks) before the first probe of words that other workgroups
// publish at about the time this one starts waiting.  A probe issued at once
// would almost surely come back without them, a coherent load takes about a
// microsecond, and many such early probes at once slow the exchange for all
// (measured: with 8-vector groups a head's y and partial-logit gathers each
// take about 0.3 to 0.5 us less with this delay than with none).
#define WR_POLL_DELAY 12
// The owned partials stay in the group's L2 (leads_share_xcd): their first
// probe waits less (measured at 64 utterances: 6 x 64 clocks 1.6% faster
// than 12, and 0.5% faster than 2).
#define WR_OWN_DELAY 6

// Wait until the N words base + off(k) carry `tag`, storing each value with
// put(k, value) as it arrives (LDS, not registers).  The addresses are
// rebuilt in every round from an opaque base, so only the N words in flight
// occupy registers.
template <int N, class O, class F>
__device__ __forceinline__ bool poll_put(const xw* base, O off, F put, uint32_t tag, const BatchArgs& a,
                                         uint32_t need = ~0u) {
  static_assert(N <= 32, "one pending bit per word");
  uint32_t pending = (N >= 32 ? ~0u : (1u << N) - 1u) & need;
  WaitBudget wb{wr_clock(), 0};
  for (;;) {
    const xw* b = opaque(base);
    xw w[N];
#pragma unroll
    for (int k = 0; k < N; ++k) w[k] = (pending >> k & 1u) ? xpeek(b + off(k)) : 0;
#pragma unroll
    for (int k = 0; k < N; ++k)
      if ((pending >> k & 1u) && xok(w[k], tag)) {
        put(k, xval(w[k]));
        pending &= ~(1u << k);
      }
    if (!pending) return true;
    if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
}

// poll_put over N pairs of adjacent words read as 64-bit accesses:
// put(k, first, second) for pair k at base + off(k) (off even).
template <int N, class O, class F>
__device__ __forceinline__ bool poll_put2(const xw* base, O off, F put, uint32_t tag, const BatchArgs& a) {
  static_assert(N <= 32, "one pending bit per pair");
  uint32_t pending = N >= 32 ? ~0u : (1u << N) - 1u;   // (a 32-bit shift by 32 is undefined)
  WaitBudget wb{wr_clock(), 0};
  for (;;) {
    const xw* b = opaque(base);
    uint64_t w[N];
#pragma unroll
    for (int k = 0; k < N; ++k) w[k] = (pending >> k & 1u) ? xpeek2(b + off(k)) : 0;
#pragma unroll
    for (int k = 0; k < N; ++k)
      if ((pending >> k & 1u) && xok2(w[k], tag)) {
        put(k, xval((xw)w[k]), xval((xw)(w[k] >> 32)));
        pending &= ~(1u << k);
      }
    if (!pending) return true;
    if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
}

// Drawn samples for the subscale context cross groups, whose heads and units
// are not chained step by step to each other: a sample word carries the
// sample (16 bits) and the low 16 bits of its tag, in one of SS slots chosen
// by the tag modulo SS.  Every lane publishes a word at every step, idle
// lanes included, and every unit waits for every lane's word of its
// utterance(s), so a head writing the samples of step s has seen the gates
// of its units for step s, which had waited for every lane's samples of step
// s - 1 - A, whose heads had seen their units finish step s - 2 - A.  No
// reader still waits for samples older than step s - 1 - 2 A, and SS >=
// 2 A + 2 slots keep the writer off them.  (Were idle lanes skipped, nothing
// would wait for a group whose lanes are all idle, and its units could fall
// any number of steps behind.)
__device__ __forceinline__ void spub(xw* slots, int L, int SS, int v, uint32_t tag, int sample) {
  __hip_atomic_store(slots + (tag & (SS - 1)) * L + v, (tag & 0xffffu) << 16 | (uint32_t)sample, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool wait_sample(const xw* slots, int L, int SS, int v, uint32_t tag, int* sample,
                                            const BatchArgs& a) {
  const xw* p = slots + (tag & (SS - 1)) * L + v;
  WaitBudget wb{wr_clock(), 0};
  for (;;) {
    const xw w = xpeek(p);
    if ((w >> 16) == (tag & 0xffffu)) {
      *sample = (int)(w & 0xffffu);
      return true;
    }
    if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
}

// ------------------------------------------------------------------ head role
// FL: the synchronization floor of the launch (every exchange, wait, barrier
// and sample word of the step, none of its arithmetic: no products, gates or
// draws; values published as zero).
template <int KH, bool CTX, int L, bool LAG, bool FL>
__device__ __forceinline__ void bhead_role(const BatchArgs& a, int g, int j, unsigned char* lds) {
  constexpr int KT = 2 * KH;
  constexpr int NH = KH;
  const BatchPlan& P = a.P;
  const int H = P.H, Hh = P.Hh;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  unsigned char* imc = lds;                        // y_c operand image [KT]
  unsigned char* imf = imc + KT * WR_FRAG;         // y_f operand image [KT]
  unsigned char* imo = imf + KT * WR_FRAG;         // relu(first layer) image [2]
  float* op = (float*)(imo + 2 * WR_FRAG);         // [2][L][64] first-layer partials
  float* zs = op + 2 * L * 64;                     // [L][256] logit sums over the heads
  float* zk = zs + L * 256;                        // [L][256] logits of the last draws
  float* hcs = zk + L * 256;                       // [L][448] coarse half of h (= y_c)
  float* hfs = hcs + L * 448;                      // [L][448] fine half of h (= y_f)
  float* gv = hfs + L * 448;                       // [4L][448] staged pre-activations and e-gate bias of the gate threads
  int64_t* cbo = (int64_t*)(gv + 4 * L * 448);    // [L] bias + conditioning row offsets of this step
  int* misc = (int*)(cbo + L);                     // [0] abort, [8+b] c_t, [16+b] c_prev, [24+b] f_prev,
                                                   // [48+b] step - position of vector b
  float* fmisc = (float*)(misc + 32);              // [b] lse_c, [8+b] z_c[c] of vector b
  float2* uni = (float2*)(misc + 64);              // [2][L][64] (u_c, u_f) of a batch of 64 steps
  int* tgt = (int*)(uni + 2 * L * 64);             // [2][L][64] teacher-forcing targets
  float* gvf = (float*)(tgt + 2 * L * 64);         // ALL: [4L][448] the fine half's words (as gv), read with the coarse

  const int v0 = g * L;                            // first vector of this group
  for (int i = tid; i < (2 * KT + 2) * WR_FRAG / 16; i += WR_THREADS) ((uint4*)lds)[i] = uint4{0, 0, 0, 0};
  bf16x8 W1[KH], W3[KH], W2[4], W4[4];
  {
    const uint4* src = a.hw + ((size_t)(j * 8 + wave) * P.hw_frags) * 64 + lane;
#pragma unroll
    for (int i = 0; i < KH; ++i) W1[i] = __builtin_bit_cast(bf16x8, src[(size_t)i * 64]);
#pragma unroll
    for (int i = 0; i < KH; ++i) W3[i] = __builtin_bit_cast(bf16x8, src[(size_t)(KH + i) * 64]);
#pragma unroll
    for (int i = 0; i < 4; ++i) W2[i] = __builtin_bit_cast(bf16x8, src[(size_t)(2 * KH + i) * 64]);
#pragma unroll
    for (int i = 0; i < 4; ++i) W4[i] = __builtin_bit_cast(bf16x8, src[(size_t)(2 * KH + 4 + i) * 64]);
  }
  const int u = tid;
  const bool gate = u < Hh;
  const bool mine = (unsigned)(u - 64 * j) < 64u;   // unit in this head's slice of y
  // With 8 vectors (SLICE) a head evaluates the gates of its own 64 units
  // only, one (unit, vector) pair per thread, and the heads exchange their
  // slices of y; with fewer vectors every head evaluates every unit of every
  // vector itself (thread u: unit u).
  constexpr bool SLICE = L == 8;
  constexpr int HH = 64 * KH;                       // Hh
  const int su = 64 * j + (tid >> 3), sb = tid & 7; // SLICE: unit and vector of this thread
  const int gu = SLICE ? su : u;                    // unit whose I* columns this thread holds
  float ic[3][2], ifn[3][3];
  if (SLICE || gate) {
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      ic[q][0] = a.Iw[3 * (q * H + gu) + 0];
      ic[q][1] = a.Iw[3 * (q * H + gu) + 1];
      ifn[q][0] = a.Iw[3 * (q * H + Hh + gu) + 0];
      ifn[q][1] = a.Iw[3 * (q * H + Hh + gu) + 1];
      ifn[q][2] = a.Iw[3 * (q * H + Hh + gu) + 2];
    }
  }
  if (gate) {
    for (int b = 0; b < L; ++b) {
      const int vb = min(v0 + b, a.S - 1);
      hcs[b * 448 + u] = a.h_in ? a.h_in[(size_t)vb * H + u] : 0.0f;
      hfs[b * 448 + u] = a.h_in ? a.h_in[(size_t)vb * H + Hh + u] : 0.0f;
    }
  }
  // relu thread: vector rb, row rr of this head's 64 first-layer rows
  const int rb = tid >> 6, rr = tid & 63;
  const float b1r = a.b1[j * 64 + rr], b3r = a.b3[j * 64 + rr];
  // draw wave w draws vector w: class biases of its 4 classes per lane
  const float4 b2l = *(const float4*)(a.b2 + 4 * lane);
  const float4 b4l = *(const float4*)(a.b4 + 4 * lane);
  if (tid < L) {
    const int vb = min(v0 + tid, a.S - 1);
    cbo[tid] = cb_offset<LAG>(a, vb, 0);
    misc[0] = 0;
    misc[16 + tid] = a.c_in ? a.c_in[vb] : 128;
    misc[24 + tid] = a.f_in ? a.f_in[vb] : 0;
    misc[8 + tid] = misc[16 + tid];
    misc[48 + tid] = LAG ? (int)(((v0 + tid) % a.B) * (a.F + 1 + a.A) - a.t0) : 0;   // position: t - misc[48 + tid]
  }
  xw* X = a.xc + (size_t)g * P.x_words;
  xw* YC = X + P.x_yc;
  xw* YF = X + P.x_yf;
  xw* PCo = X + P.x_pc + (size_t)j * L * 256;
  xw* PFo = X + P.x_pf + (size_t)j * L * 256;
  const xw* PC = X + P.x_pc;
  const xw* PF = X + P.x_pf;
  const int rt = wave & 3, kc = wave >> 2;
  const int bl0 = 2 * (lane >> 4);                 // vectors of this lane's MFMA results: bl0, bl0 + 1

  auto first_layer = [&](const bf16x8* W, const unsigned char* img, float bias) {
    if (!FL) {
      f32x4 acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < KH; i += 2) {
        acc0 = mfma(afrag(img, kc * KH + i), W[i], acc0);
        if (i + 1 < KH) acc1 = mfma(afrag(img, kc * KH + i + 1), W[i + 1], acc1);
      }
      const int r = 16 * rt + (lane & 15);
      if (bl0 < L) {                                // lanes of vectors past L hold rows of zero inputs
        op[(kc * L + bl0) * 64 + r] = mfma_row(acc0) + mfma_row(acc1);
        op[(kc * L + bl0 + 1) * 64 + r] = mfma_row_hi(acc0) + mfma_row_hi(acc1);
      }
    }
    __syncthreads();
    if (!FL && rb < L)
      aput(imo + (rr >> 5) * WR_FRAG, rr & 31, wr_relu((op[rb * 64 + rr] + op[(L + rb) * 64 + rr]) + bias), rb);
    __syncthreads();
  };
  // class tiles 2*wave, 2*wave+1 over this head's 64 columns, for all vectors
  bool lx = false;   // the group's heads share one XCD: partials and classes into its L2
  auto second_layer = [&](const bf16x8* W, xw* dst, uint32_t tag) {
    f32x4 A = {0, 0, 0, 0}, B = {0, 0, 0, 0};
    if (!FL) {
      const bf16x8 x0 = afrag(imo, 0), x1 = afrag(imo, 1);
      A = mfma(x0, W[0], A);
      B = mfma(x0, W[2], B);
      A = mfma(x1, W[1], A);
      B = mfma(x1, W[3], B);
    }
    const int c0 = 32 * wave + (lane & 15);
    if (bl0 < L) {
      xpub_l(dst + bl0 * 256 + c0, tag, mfma_row(A), lx);
      xpub_l(dst + (bl0 + 1) * 256 + c0, tag, mfma_row_hi(A), lx);
      xpub_l(dst + bl0 * 256 + c0 + 16, tag, mfma_row(B), lx);
      xpub_l(dst + (bl0 + 1) * 256 + c0 + 16, tag, mfma_row_hi(B), lx);
    }
  };
  // Vector ownership.  With 8 vectors per group head j draws the vectors j,
  // j + NH, ... (slot q: vector j + NH q) and every other head learns their
  // classes from one word each: only the owner sums a vector's partial
  // logits, so a head reads 1/NH of the partials.  With up to 4 vectors
  // (ALL) every head sums and draws every vector (slot q: vector q): the
  // partials of all of them are no more words per thread than an owner's
  // share of 8, and no class words have to travel.
  constexpr bool ALL = L <= 4;
  constexpr int OV = ALL ? L : (L + NH - 1) / NH;   // most vectors a head draws
  constexpr int SP = (OV + 1) / 2;                  // drawn slots per gathering thread
  const int nown = ALL ? L : (L - j + NH - 1) / NH; // vectors this head draws
  auto vec = [&](int q) { return ALL ? q : j + NH * q; };   // vector of slot q
  // Sums over the heads, in head order, of the owned vectors' partials:
  // thread (class v, parity s) reads slots s, s + 2, ... of every head (all
  // words in flight at once, the first probe after WR_POLL_DELAY), re-reading
  // only words without the step's tag.
  auto gather_own = [&](const xw* src, uint32_t tag) {
    __builtin_amdgcn_s_sleep(WR_OWN_DELAY);
    const int v = tid & 255, sp = tid >> 8;
    // word k (< SP NH): head k % NH, slot sp + 2 (k / NH); staged in gv (free here)
    float* stage = gv + tid;                        // [SP NH][512]
    uint32_t need = 0;
#pragma unroll
    for (int k = 0; k < SP * NH; ++k)
      if (sp + 2 * (k / NH) < nown) need |= 1u << k;
    if (!poll_put<SP * NH>(src + v,
                           [&](int k) { return (size_t)((k % NH) * L + vec(sp + 2 * (k / NH))) * 256; },
                           [&](int k, float x) { stage[k * WR_THREADS] = x; }, tag, a, need)) {
      misc[0] = 1;
      return;
    }
#pragma unroll
    for (int m = 0; m < SP; ++m) {
      if (sp + 2 * m >= nown) break;
      float s = 0.0f;
#pragma unroll
      for (int jj = 0; jj < NH; ++jj) s += stage[(m * NH + jj) * WR_THREADS];
      zs[(sp + 2 * m) * 256 + v] = s;
    }
  };
  // The 3L pre-activation words of gate thread u of each half and the L
  // additive terms of each half's e gate (bias + conditioning, and with
  // subscale the context term, which stays outside the reset product), staged
  // in LDS: coarse word k at gv[k * 448 + u] and the term of vector b at
  // gv[(3L + b) * 448 + u], fine ones likewise in gvf.  The units publish
  // both halves at once, so all 4L word pairs are polled together at the
  // start of the step: the fine gates wait for nothing but c_t.
  const bool trg = g == 0 && j == 0 && tid == 0;            // a gate thread (tracing)
  auto read_gates = [&](uint32_t tag, int64_t t) {
#pragma unroll
    for (int b = 0; b < L; ++b) {
      gv[(3 * L + b) * 448 + u] = a.cb[cbo[b] + 2 * H + u];
      gvf[(3 * L + b) * 448 + u] = a.cb[cbo[b] + 2 * H + Hh + u];
    }
    if (trg) trace_at(a, t, 13);
    // pair k: half k / HP; in a half, the context pairs (vectors 2r, 2r + 1) and
    // then the gate pairs (gate q, vectors b, b + 1) of unit u
    constexpr int XP = CTX ? L / 2 : 0, HP = XP + 3 * L / 2;
    if (!poll_put2<2 * HP>((const xw*)X,
                           [&](int k) -> size_t {
                             const int h = k / HP, r = k % HP;
                             if (r < XP) return (size_t)(h ? P.x_xf : P.x_xc) + (size_t)u * L + 2 * r;
                             const int q = (r - XP) / (L / 2), b = 2 * ((r - XP) % (L / 2));
                             return (size_t)(h ? P.x_gf : P.x_ga) + (size_t)q * Hh * L + (size_t)u * L + b;
                           },
                           [&](int k, float x0, float x1) {
                             const int h = k / HP, r = k % HP;
                             float* gw = h ? gvf : gv;
                             if (r < XP) {
                               gw[(3 * L + 2 * r) * 448 + u] += x0;
                               gw[(3 * L + 2 * r + 1) * 448 + u] += x1;
                             } else {
                               const int q = (r - XP) / (L / 2), b = 2 * ((r - XP) % (L / 2));
                               gw[(3 * b + q) * 448 + u] = x0;
                               gw[(3 * b + 3 + q) * 448 + u] = x1;
                             }
                           },
                           tag, a))
      misc[0] = 1;
  };
  xw* CC = X + P.x_cc;                              // drawn coarse classes [L]
  xw* CF = X + P.x_cf;                              // drawn fine classes [L]
  // SLICE: one (unit, vector) pair per thread.  Its three pre-activation
  // words, the e gate's context term (subscale) and, for the coarse half,
  // the first word unit k = tid publishes: a unit publishes its words of
  // step t + 1 only after reading all of h of step t, so once every unit's
  // word has arrived this head may replace its slice of y of step t.  Then
  // the gates, this head's slice of y, and the other slices from their heads.
  // The classes of the thread's vector travel with the same poll: c_{t-1} and
  // f_{t-1} with the coarse words (from step 1 on), c_t with the fine words.
  int cprev = 0, fprev = 0, ccur = 0;               // SLICE: classes of vector sb
  size_t uflag = 0;
  if (SLICE && tid < P.NU) {
    const int tile = tid * WR_BUCT, gt = tile / (HH / 16);
    uflag = P.x_ga + (size_t)(gt * HH + 16 * (tile % (HH / 16))) * L;
  }
  auto slice_gates = [&](bool fine, uint32_t tag, int64_t t, uint32_t actm) {
    const float cb = a.cb[cbo[sb] + 2 * H + (fine ? HH : 0) + su];
    const size_t go = (fine ? P.x_gf : P.x_ga) + (size_t)su * L + sb;
    const size_t xo = (fine ? P.x_xf : P.x_xc) + (size_t)su * L + sb;
    // words 0-2 gates, 3 context term, 4 unit flag, 5 c (fine: c_t; coarse: c_{t-1}), 6 f_{t-1}
    uint32_t pending = 7u | (CTX ? 8u : 0u) | (!fine && tid < P.NU ? 16u : 0u) | (fine ? 32u : t > 0 ? 96u : 0u);
    float gw[7] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    const size_t co = P.x_cc + sb, fo = P.x_cf + sb;
    WaitBudget wb{wr_clock(), 0};
    for (;;) {
      const xw* xb = opaque((const xw*)X);
      xw w[7];
#pragma unroll
      for (int k = 0; k < 7; ++k)
        w[k] = (pending >> k & 1u) ? xpeek(xb + (k < 3 ? go + (size_t)k * HH * L : k == 3 ? xo : k == 4 ? uflag : k == 5 ? co : fo)) : 0;
#pragma unroll
      for (int k = 0; k < 7; ++k)
        if ((pending >> k & 1u) && xok(w[k], k >= 5 && !fine ? tag - 1u : tag)) {
          gw[k] = xval(w[k]);
          pending &= ~(1u << k);
        }
      if (!pending) break;
      if (!wait_ok(wb, a.err, a.limit, a.err)) {
        misc[0] = 1;
        return;
      }
    }
    if (trg) trace_at(a, t, fine ? 12 : 11);
    if (FL) {                                       // the exchange alone: own slice out, the others in
      xpub((fine ? YF : YC) + sb * HH + su, tag, 0.0f);
      uint32_t own = 0;
#pragma unroll
      for (int m = 0; m < KH; ++m)
        if ((tid + WR_THREADS * m) % HH / 64 == j) own |= 1u << m;
      __builtin_amdgcn_s_sleep(WR_POLL_DELAY);
      if (!poll_put<KH>(fine ? YF : YC, [&](int m) { return (size_t)(tid + WR_THREADS * m); },
                        [&](int, float) {}, tag, a, ~own))
        misc[0] = 1;
      return;
    }
    if (fine) ccur = (int)gw[5];
    else if (t > 0) {
      cprev = (int)gw[5];
      fprev = (int)gw[6];
    }
    const float cbe = cb + gw[3];
    const float x0 = fscale(cprev), x1 = fscale(fprev);
    float pu, pr, pe;
    if (fine) {
      const float x2 = fscale(ccur);
      pu = __builtin_fmaf(ifn[0][2], x2, __builtin_fmaf(ifn[0][1], x1, ifn[0][0] * x0));
      pr = __builtin_fmaf(ifn[1][2], x2, __builtin_fmaf(ifn[1][1], x1, ifn[1][0] * x0));
      pe = __builtin_fmaf(ifn[2][2], x2, __builtin_fmaf(ifn[2][1], x1, ifn[2][0] * x0));
    } else {
      pu = __builtin_fmaf(ic[0][1], x1, ic[0][0] * x0);
      pr = __builtin_fmaf(ic[1][1], x1, ic[1][0] * x0);
      pe = __builtin_fmaf(ic[2][1], x1, ic[2][0] * x0);
    }
    const float uu = fsig(gw[0] + pu);
    const float rg = fsig(gw[1] + pr);
    const float e = ftanh(__builtin_fmaf(rg, gw[2], pe + cbe));
    float* hs = (fine ? hfs : hcs) + sb * 448 + su;
    const float hn = actm >> sb & 1u ? __builtin_fmaf(uu, *hs, (1.0f - uu) * e) : *hs;   // idle: state kept
    *hs = hn;
    unsigned char* img = fine ? imf : imc;
    aput(img + (su >> 5) * WR_FRAG, su & 31, xround(hn), sb);
    xw* Y = fine ? YF : YC;
    xpub(Y + sb * HH + su, tag, hn);
    // the other heads' slices: word w = tid + 512 m of y [8][Hh] (Hh / 64 per thread)
    uint32_t own = 0;
#pragma unroll
    for (int m = 0; m < KH; ++m)
      if ((tid + WR_THREADS * m) % HH / 64 == j) own |= 1u << m;
    __builtin_amdgcn_s_sleep(WR_POLL_DELAY);
    if (!poll_put<KH>(Y, [&](int m) { return (size_t)(tid + WR_THREADS * m); },
                      [&](int m, float y) {
                        const int w = tid + WR_THREADS * m, b = w / HH, c = w % HH;
                        aput(img + (c >> 5) * WR_FRAG, c & 31, y, b);
                      },
                      tag, a, ~own))
      misc[0] = 1;
  };
  const int bw = vec(wave);                         // vector (in the group) drawn by this wave, if wave < nown
  const int vw = min(v0 + bw, a.S - 1);
  const size_t ob = obase(a, vw);
  auto fill_batch = [&](int64_t t, int buf) {       // wave w: uniforms / targets of its owned vector
    const int64_t s = t + lane, p = vpos<LAG>(a, vw, s);
    if (s < a.T && p >= 0 && p < a.rows) {
      float uc, uf;
      wr_uniforms(a.seed, (uint64_t)vw, (uint64_t)((LAG ? 0 : a.t0) + p), &uc, &uf);
      uni[(buf * L + wave) * 64 + lane] = float2{uc, uf};
      tgt[(buf * L + wave) * 64 + lane] = a.target ? a.target[ob + (size_t)a.B * p] : 0;
    }
  };
  if (wave < nown) fill_batch(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (SLICE) {
    cprev = misc[16 + sb];
    fprev = misc[24 + sb];
  }
  const bool trw = g == 0 && j == 0 && tid == WR_THREADS - 64;
  const bool own = wave < nown;                     // this wave draws an owned vector
  const bool writer = own && (!ALL || bw % NH == j); // ... and writes its outputs (one head per vector)
  const bool live = writer && v0 + bw < a.S;       // ... of a vector in use
  if (WR_LOCAL_XCHG) lx = leads_share_xcd(X + P.x_xcc, P.NH, j, misc + 1, a);

  for (int64_t t = 0; t < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    if (trw) trace_at(a, t, 0);
    // bit b: vector b is at one of its lane's positions this step (always so
    // for lockstep rows; with a horizon lane b runs position t - misc[48 + b])
    uint32_t actm = ~0u;
    if (LAG) {
#pragma unroll
      for (int b = 0; b < L; ++b) {
        const int64_t p = t - misc[48 + b];
        if (p < 0 || p >= a.rows) actm &= ~(1u << b);
      }
    }
    const int bs = (int)((t >> 6) & 1) * L * 64 + wave * 64 + (int)(t & 63);   // draw wave's batch slot
    if (own && (t & 63) == 0) fill_batch(t + 64, (int)(((t >> 6) + 1) & 1));
    // (1) coarse gates of every unit and vector: the pre-activation words of
    // thread u (both halves with up to 4 vectors) are polled together and
    // staged in LDS, then one vector at a time
    if (SLICE) {
      slice_gates(false, tag, t, actm);
    } else if (gate) {
      read_gates(tag, t);
      if (trg) trace_at(a, t, 11);
#pragma unroll 2
      for (int b = 0; b < L; ++b) {
        if (FL) {
          if (mine) xpub(YC + b * Hh + u, tag, 0.0f);
          continue;
        }
        const float cbe = gv[(3 * L + b) * 448 + u];
        const float x0 = fscale(misc[16 + b]), x1 = fscale(misc[24 + b]);
        const float uu = fsig(gv[(3 * b) * 448 + u] + __builtin_fmaf(ic[0][1], x1, ic[0][0] * x0));
        const float rg = fsig(gv[(3 * b + 1) * 448 + u] + __builtin_fmaf(ic[1][1], x1, ic[1][0] * x0));
        const float e = ftanh(
            __builtin_fmaf(rg, gv[(3 * b + 2) * 448 + u], __builtin_fmaf(ic[2][1], x1, ic[2][0] * x0) + cbe));
        const float hn = actm >> b & 1u ? __builtin_fmaf(uu, hcs[b * 448 + u], (1.0f - uu) * e)
                                        : hcs[b * 448 + u];   // an idle lane keeps its state
        hcs[b * 448 + u] = hn;
        aput(imc + (u >> 5) * WR_FRAG, u & 31, hn, b);
        if (mine) xpub(YC + b * Hh + u, tag, hn);   // this head's slice, for the units
      }
    }
    __syncthreads();
    if (misc[0]) return;
    if (trw) trace_at(a, t, 1);
    // (2) O1 rows, relu, O2 columns -> partial coarse logits of 8 vectors
    first_layer(W1, imc, b1r);
    second_layer(W2, PCo, tag);
    if (trw) trace_at(a, t, 3);
    // (3) the owned vectors' sums over the heads, their coarse draws (wave w:
    // slot w), then every vector's class from its owner
    gather_own(PC, tag);
    __syncthreads();
    if (misc[0]) return;
    if (trw) trace_at(a, t, 4);
    if (own) {
      float lse;
      const int forced = a.target ? (tgt[bs] >> 8) : -1;
      const int c = FL ? 0 : draw_wave<false>(zs + wave * 256, nullptr, b2l, uni[bs].x, forced, zk + wave * 256,
                                              a.nll_out ? &lse : nullptr);
      const int64_t pw = LAG ? t - misc[48 + bw] : t;   // this vector's position; an idle lane keeps its classes
      const bool act = actm >> bw & 1u;
      if (live && act && a.zc_out)
        *(float4*)(a.zc_out + (ob + (size_t)a.B * pw) * WR_CLASSES + 4 * lane) =
            *(const float4*)(zk + wave * 256 + 4 * lane);
      if (lane == 0) {
        int cw = c;                                 // the class word: an idle lane's last class
        if (act) misc[8 + bw] = c;
        else cw = misc[8 + bw];
        if (!ALL) xpub_l(CC + bw, tag, (float)cw, lx);
        if (a.nll_out) {
          fmisc[wave] = lse;
          fmisc[8 + wave] = zk[wave * 256 + c];
        }
      }
    }
    __syncthreads();
    if (trw) trace_at(a, t, 5);
    // (4) fine gates with c_t
    if (SLICE) {
      slice_gates(true, tag, t, actm);
    } else if (gate) {
      if (trg) trace_at(a, t, 12);                 // (the fine words came with the coarse ones)
#pragma unroll 2
      for (int b = 0; b < L; ++b) {
        if (FL) {
          if (mine) xpub(YF + b * Hh + u, tag, 0.0f);
          continue;
        }
        const float cbe = gvf[(3 * L + b) * 448 + u];
        const float x0 = fscale(misc[16 + b]), x1 = fscale(misc[24 + b]), x2 = fscale(misc[8 + b]);
        const float uu = fsig(gvf[(3 * b) * 448 + u] +
                              __builtin_fmaf(ifn[0][2], x2, __builtin_fmaf(ifn[0][1], x1, ifn[0][0] * x0)));
        const float rg = fsig(gvf[(3 * b + 1) * 448 + u] +
                              __builtin_fmaf(ifn[1][2], x2, __builtin_fmaf(ifn[1][1], x1, ifn[1][0] * x0)));
        const float e = ftanh(__builtin_fmaf(
            rg, gvf[(3 * b + 2) * 448 + u],
            __builtin_fmaf(ifn[2][2], x2, __builtin_fmaf(ifn[2][1], x1, ifn[2][0] * x0)) + cbe));
        const float hn = actm >> b & 1u ? __builtin_fmaf(uu, hfs[b * 448 + u], (1.0f - uu) * e)
                                        : hfs[b * 448 + u];
        hfs[b * 448 + u] = hn;
        aput(imf + (u >> 5) * WR_FRAG, u & 31, hn, b);
        if (mine) xpub(YF + b * Hh + u, tag, hn);
      }
    }
    __syncthreads();
    if (misc[0]) return;
    if (trw) trace_at(a, t, 6);
    // (5) O3 rows, relu, O4 columns -> partial fine logits
    first_layer(W3, imf, b3r);
    second_layer(W4, PFo, tag);
    if (trw) trace_at(a, t, 8);
    // (6) the owned vectors' fine sums and draws, then every vector's class
    gather_own(PF, tag);
    __syncthreads();
    if (misc[0]) return;
    if (trw) trace_at(a, t, 9);
    if (own) {
      float lse;
      const int forced = a.target ? (tgt[bs] & 255) : -1;
      const int f = FL ? 0 : draw_wave<false>(zs + wave * 256, nullptr, b4l, uni[bs].y, forced, zk + wave * 256,
                                              a.nll_out ? &lse : nullptr);
      const int c = misc[8 + bw];
      const int64_t pw = LAG ? t - misc[48 + bw] : t;
      const bool act = actm >> bw & 1u;
      if (live && act && a.zf_out)
        *(float4*)(a.zf_out + (ob + (size_t)a.B * pw) * WR_CLASSES + 4 * lane) =
            *(const float4*)(zk + wave * 256 + 4 * lane);
      if (lane == 0) {
        int fw = f;
        if (SLICE) {                                // the owner's record (final state)
          if (act) misc[24 + bw] = f;
          else fw = misc[24 + bw];
        }
        if (!ALL) xpub_l(CF + bw, tag, (float)fw, lx);
        // for later contexts; an idle lane publishes a word too (value unused)
        if (a.ux && writer) spub(X + P.x_sp, L, P.SS, bw, tag, act ? 256 * c + f : 0);
        if (live && act) {
          if (a.out) a.out[ob + (size_t)a.B * pw] = (uint16_t)(256 * c + f);
          if (a.nll_out)
            a.nll_out[ob + (size_t)a.B * pw] = (fmisc[wave] - fmisc[8 + wave]) + (lse - zk[wave * 256 + f]);
        }
        if (ALL) {                                  // this head's own record of the vector's classes
          if (act) {
            misc[16 + bw] = c;
            misc[24 + bw] = f;
          }
          if (t + 1 < a.T) cbo[bw] = cb_offset<LAG>(a, min(v0 + bw, a.S - 1), t + 1);
        }
      }
    }
    if (SLICE && tid < L && t + 1 < a.T) cbo[tid] = cb_offset<LAG>(a, min(v0 + tid, a.S - 1), t + 1);
    __syncthreads();
    if (trw) trace_at(a, t, 10);
  }
  if (SLICE && a.h_out && v0 + sb < a.S) {          // each head its own slice
    a.h_out[(size_t)(v0 + sb) * H + su] = hcs[sb * 448 + su];
    a.h_out[(size_t)(v0 + sb) * H + Hh + su] = hfs[sb * 448 + su];
  }
  if (j == 0) {
    if (a.h_out && gate && !SLICE)
      for (int b = 0; b < L; ++b)
        if (v0 + b < a.S) {
          a.h_out[(size_t)(v0 + b) * H + u] = hcs[b * 448 + u];
          a.h_out[(size_t)(v0 + b) * H + Hh + u] = hfs[b * 448 + u];
        }
    if (tid < L && v0 + tid < a.S && !SLICE) {
      if (a.c_out) a.c_out[v0 + tid] = (uint8_t)misc[16 + tid];
      if (a.f_out) a.f_out[v0 + tid] = (uint8_t)misc[24 + tid];
    }
  }
  if (SLICE && lane == 0 && live) {                 // the owner: last classes of its vectors
    if (a.c_out) a.c_out[v0 + bw] = (uint8_t)misc[8 + bw];
    if (a.f_out) a.f_out[v0 + bw] = (uint8_t)misc[24 + bw];
  }
}

// ------------------------------------------------------------------ unit role
// Wave q < 4 owns coarse row tile 4k + q, wave 4 + q fine row tile 4k + q;
// each lane of a wave's result holds two vectors of one row, which it
// publishes (with bias + conditioning for the u and r gates).
template <int KH, bool CTX, int L, bool LAG, bool FL>
__device__ __forceinline__ void bunit_role(const BatchArgs& a, int g, int k, unsigned char* lds) {
  constexpr int KT = 2 * KH;
  const BatchPlan& P = a.P;
  const int H = P.H, Hh = P.Hh;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const bool fw = wave >= 4;
  const int q = wave & 3;
  const unsigned char* WL = lds + (fw ? WR_BUCT * KT + q * KT : q * KT) * WR_FRAG;   // this wave's LDS half
  unsigned char* img = lds + P.u_lds_w;                                             // [2KT] operand image
  unsigned char* cimg = img + 2 * KT * WR_FRAG;                                     // [KX] context image
  int* hist = (int*)(cimg + P.KX * WR_FRAG);          // [utterance slot][HC]: sample q at q % HC
  int* misc = hist + P.RING;
  const int HC = LAG ? P.HC : 256, HCm = HC - 1;   // (256 always holds a lockstep context)
  const int tile = k * WR_BUCT + q;
  const int gt = tile / (Hh / 16), i = 16 * (tile % (Hh / 16)) + (lane & 15);
  const int row = gt * H + (fw ? Hh : 0) + i;                  // R row of this lane
  const int bl0 = 2 * (lane >> 4);
  const int v0 = g * L;
  xw* X = a.xc + (size_t)g * P.x_words;
  xw* dst = X + (fw ? P.x_gf : P.x_ga) + (size_t)(gt * Hh + i) * L + bl0;   // vectors bl0, bl0 + 1
  {
    const uint4* src = a.uw + (size_t)k * (P.u_lds_w / 16);
    for (int x = tid; x < P.u_lds_w / 16; x += WR_THREADS) ((uint4*)lds)[x] = src[x];
    for (int x = tid; x < (2 * KT + P.KX) * WR_FRAG / 16; x += WR_THREADS) ((uint4*)img)[x] = uint4{0, 0, 0, 0};
    if (tid == 0) misc[0] = 0;
  }
  bf16x8 WX[CTX ? 8 : 1];                              // context-projection fragments of this wave's tile
  if (CTX) {
    const uint4* src = a.ux + ((size_t)(k * 8 + wave) * P.KX) * 64 + lane;
#pragma unroll
    for (int x = 0; x < (CTX ? 8 : 0); ++x)
      if (x < P.KX) WX[x] = __builtin_bit_cast(bf16x8, src[(size_t)x * 64]);
  }
  bf16x8 WR[KT];
  {
    const uint4* src = a.ur + ((size_t)(k * 8 + wave) * KT) * 64 + lane;
#pragma unroll
    for (int x = 0; x < KT; ++x) WR[x] = __builtin_bit_cast(bf16x8, src[(size_t)x * 64]);
  }
  __syncthreads();
  for (int x = tid; x < L * H; x += WR_THREADS) {
    const int b = x / H, col = x % H;
    const float y = a.h_in ? xround(a.h_in[(size_t)min(v0 + b, a.S - 1) * H + col]) : 0.0f;
    aput(img + (col >> 5) * WR_FRAG, col & 31, y, b);
  }
  // A launch that starts at step t0 > 0 of a call (the call resumed) starts
  // each ring slot with what a launch from step 0 would hold there now: slot
  // sl of an utterance holds sample q = B p + z, q = sl mod HC, of the last
  // position p of lane z = sl mod B (B divides HC) made before step t0.
  if (CTX && !(LAG && a.ctab) && a.prev && a.t0 > 0) {
    const int per = HC / a.B;
    const int u0 = v0 / a.B, nu = a.B >= L ? 1 : L / a.B;
    for (int x = tid; x < nu * HC; x += WR_THREADS) {
      const int uo = x / HC, sl = x % HC, z = sl % a.B, r = (sl - z) / a.B;
      int y = 0;
      if ((u0 + uo) * a.B < a.S) {
        int64_t pz = LAG ? a.t0 - (int64_t)z * (a.F + 1 + a.A) : a.t0;   // lane z's positions made so far
        if (pz > a.rows) pz = a.rows;
        if (pz > 0) {
          const int64_t p = pz - 1 - ((pz - 1 - r) % per + per) % per;   // last such p with p = r mod per
          if (p >= 0) y = a.prev[(size_t)(u0 + uo) * a.B * a.rows + (size_t)a.B * p + z];
        }
      }
      hist[uo * HC + sl] = y;
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  f32x4 acc0, acc1;
  // coarse inputs (image tiles 0 .. KT-1): coarse waves from LDS, fine waves from VGPRs
  auto phase_c = [&]() {
    acc0 = f32x4{0, 0, 0, 0};
    acc1 = f32x4{0, 0, 0, 0};
    if (FL) return;
#pragma unroll
    for (int x = 0; x < KT; x += 2) {
      const bf16x8 w0 = fw ? WR[x] : *(const bf16x8*)(WL + x * WR_FRAG + lane * 16);
      acc0 = mfma(afrag(img, x), w0, acc0);
      if (x + 1 < KT) {
        const bf16x8 w1 = fw ? WR[x + 1] : *(const bf16x8*)(WL + (x + 1) * WR_FRAG + lane * 16);
        acc1 = mfma(afrag(img, x + 1), w1, acc1);
      }
    }
  };
  // fine inputs (image tiles KT .. 2KT-1)
  auto phase_f = [&]() {
    if (FL) return;
#pragma unroll
    for (int x = 0; x < KT; x += 2) {
      const bf16x8 w0 = fw ? *(const bf16x8*)(WL + x * WR_FRAG + lane * 16) : WR[x];
      acc0 = mfma(afrag(img, KT + x), w0, acc0);
      if (x + 1 < KT) {
        const bf16x8 w1 = fw ? *(const bf16x8*)(WL + (x + 1) * WR_FRAG + lane * 16) : WR[x + 1];
        acc1 = mfma(afrag(img, KT + x + 1), w1, acc1);
      }
    }
  };
  f32x4 xa0 = {0, 0, 0, 0}, xa1 = {0, 0, 0, 0};        // context term of e-gate rows
  xw* dstx = X + (fw ? P.x_xf : P.x_xc) + (size_t)i * L + bl0;
  // With the context formed ahead (A > 0, or read from a table) it is built
  // at the start of a step, before h arrives, into its own sums for every row.
  const bool table = CTX && LAG && a.ctab;
  const bool ahead = CTX && LAG && (a.A > 0 || table);
  auto publish = [&](uint32_t tag, float cb0, float cb1) {
    if (bl0 >= L) return;                               // rows of vectors past L: zero inputs, not published
    if (ahead && gt < 2) {
      cb0 += mfma_row(xa0) + mfma_row(xa1);
      cb1 += mfma_row_hi(xa0) + mfma_row_hi(xa1);
    }
    xpub2(dst, tag, (mfma_row(acc0) + mfma_row(acc1)) + cb0, (mfma_row_hi(acc0) + mfma_row_hi(acc1)) + cb1);
    if (CTX && gt == 2) xpub2(dstx, tag, mfma_row(xa0) + mfma_row(xa1), mfma_row_hi(xa0) + mfma_row_hi(xa1));
  };
  // Subscale context (Sec. 4): the samples drawn at step t - A by the lanes
  // of every utterance of this group join the ring; vector b's context for
  // step t + 1 is Dx/2 samples as (c, f) scaled: lockstep, the ones before
  // its own sample, zero for samples of row t + 1 or before the start; with
  // horizon F (Sec. 4.2) Dx/4 before and Dx/4 after its own, zero unless an
  // earlier sub-tensor made it at a position up to p + F.  Sub-tensor z runs
  // position p + F at step p + F + z (F + 1 + A), at most t - A for z < s,
  // so the ring holds every such sample.  Its projection joins the sums of
  // the u and r rows; for e rows it is kept apart (published on its own: it
  // is not reset-gated).
  const int ub0 = v0 / a.B;                            // first utterance of this group
  const int nut = a.B >= L ? 1 : L / a.B;              // utterances of this group
  // Table context (the conditioning CNN's output, Sec. 4.1): vector b's
  // context for step t + 1 is the table row of the position it runs there
  // (block of the vector, rows from ctab_row0 + s ctab_step on; an idle
  // lane's row clamped into the block); nothing to wait for.
  auto table_image = [&](int64_t t) {
    const int Dx = a.P.KX * 32;
    for (int x = tid; x < L * Dx; x += WR_THREADS) {
      const int b = x / Dx, col = x % Dx;
      const int vb = min(v0 + b, a.S - 1);
      int64_t r = vpos<LAG>(a, vb, t + 1) - (a.ctab_row0 + (int64_t)(vb % a.B) * a.ctab_step);
      r = r < 0 ? 0 : r >= a.ctab_rows ? a.ctab_rows - 1 : r;
      aput(cimg + (col >> 5) * WR_FRAG, col & 31, a.ctab[((size_t)vb * a.ctab_rows + r) * Dx + col], b);
    }
    __syncthreads();
  };
  auto context = [&](int64_t t) {
    if (table) {
      table_image(t);
    } else {
    const int64_t td = t - (LAG ? a.A : 0);            // the step whose samples join the ring now
    const uint32_t tag = (uint32_t)(td + 1);
    if (tid < nut * a.B && td >= 0) {                  // one thread per (utterance, lane)
      const int vv = ub0 * a.B + tid;                  // vector of that lane
      int y = 0;
      const int64_t p = vpos<LAG>(a, vv, td);          // lanes idle at step td drew nothing
      if (vv < a.S) {                                  // (but their words are waited for too)
        if (!wait_sample(a.xc + (size_t)(vv / L) * P.x_words + P.x_sp, L, P.SS, vv % L, tag, &y, a)) misc[0] = 1;
        const int64_t qn = (int64_t)a.B * (p + (LAG ? 0 : a.t0)) + tid % a.B;   // the sample's index
        if (p >= 0 && p < a.rows) hist[(tid / a.B) * HC + (int)(qn & HCm)] = y;
      }
    }
    __syncthreads();
    if (misc[0] || FL) return;                         // (the floor: the sample waits, not the context)
    const int half = a.P.KX * 16;                      // context samples per vector
    for (int x = tid; x < L * half; x += WR_THREADS) {
      const int b = x / half, jj = x % half;
      const int vb = min(v0 + b, a.S - 1), s = vb % a.B;
      const int64_t p1 = vpos<LAG>(a, vb, t + 1);           // position this vector runs next
      const int64_t n1 = (int64_t)a.B * (p1 + (LAG ? 0 : a.t0)) + s;   // the sample it makes there
      int64_t qn;
      bool seen;
      if (!LAG) {                                      // lockstep: the samples before n1 of earlier rows
        qn = n1 - 1 - jj;
        seen = qn >= 0 && qn < (int64_t)a.B * (a.t0 + t + 1);
      } else {                                         // horizon F: half before n1, half after
        const int d = jj < half / 2 ? -1 - jj : 1 + (jj - half / 2);
        qn = n1 + d;
        // q = B (p1 + dk) + z with 0 <= z < B: small integers only
        const int sd = s + d + 2 * half * a.B;         // > 0
        const int dk = sd / a.B - 2 * half, z = sd % a.B;
        seen = p1 >= 0 && p1 < a.rows && qn >= 0 && qn < (int64_t)a.B * a.rows && z < s && dk <= a.F;
      }
      float c = 0.0f, f = 0.0f;
      if (seen) {
        const int sv = hist[(vb / a.B - ub0) * HC + (int)(qn & HCm)];
        c = fscale(sv >> 8);
        f = fscale(sv & 255);
      }
      aput(cimg + ((2 * jj) >> 5) * WR_FRAG, (2 * jj) & 31, c, b);
      aput(cimg + ((2 * jj + 1) >> 5) * WR_FRAG, (2 * jj + 1) & 31, f, b);
    }
    __syncthreads();
    }
    const bool apart = gt == 2 || ahead;               // kept apart from the products of h
    f32x4 c0 = apart ? f32x4{0, 0, 0, 0} : acc0, c1 = apart ? f32x4{0, 0, 0, 0} : acc1;
#pragma unroll
    for (int x = 0; x < (CTX ? 8 : 0); x += 2) {
      if (x < P.KX) c0 = mfma(afrag(cimg, x), WX[x], c0);
      if (x + 1 < P.KX) c1 = mfma(afrag(cimg, x + 1), WX[x + 1], c1);
    }
    if (apart) {
      xa0 = c0;
      xa1 = c1;
    } else {
      acc0 = c0;
      acc1 = c1;
    }
  };
  auto cbv = [&](int b, int64_t t) {                           // u and r gates carry bias + conditioning
    return gt < 2 && b < L ? a.cb[cb_offset<LAG>(a, min(v0 + b, a.S - 1), t) + row] : 0.0f;
  };
  // Wait for one half of h of the group's vectors and write the operand
  // tiles kt0 ...: with 8 vectors (7 words per thread) lane jj of wave 0
  // first watches the last word head jj publishes, so that only 7 words per
  // wave are polled while h is not there; with fewer vectors every thread
  // polls its own words directly, the first probe after WR_POLL_DELAY.
  auto gather_half = [&](const xw* Y, uint32_t tag, int kt0) {
    if (L < 8) __builtin_amdgcn_s_sleep(WR_POLL_DELAY);
    if (L >= 8) {
      if (wave == 0) {
        const int hj = lane < P.NH ? lane : 0;
        float y;
        if (!poll_strided<1>(Y + (L - 1) * Hh + 64 * hj + 63, 0, tag, &y, a)) misc[0] = 1;
      }
      __syncthreads();
      if (misc[0]) return;
    }
    constexpr int PER = (L * 448 + WR_THREADS - 1) / WR_THREADS;   // words per thread at most
    float y[PER];
    uint32_t pending = 0;
#pragma unroll
    for (int m = 0; m < PER; ++m)
      if (tid + m * WR_THREADS < L * Hh) pending |= 1u << m;
    WaitBudget wb{wr_clock(), 0};
    while (pending) {
      xw w[PER];
#pragma unroll
      for (int m = 0; m < PER; ++m) w[m] = (pending >> m & 1u) ? xpeek(Y + tid + m * WR_THREADS) : 0;
#pragma unroll
      for (int m = 0; m < PER; ++m)
        if ((pending >> m & 1u) && xok(w[m], tag)) {
          y[m] = xval(w[m]);
          pending &= ~(1u << m);
        }
      if (pending && !wait_ok(wb, a.err, a.limit, a.err)) {
        misc[0] = 1;
        break;
      }
    }
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int x = tid + m * WR_THREADS;
      if (!FL && x < L * Hh && !(pending >> m & 1u)) {
        const int b = x / Hh, col = x % Hh;
        aput(img + (kt0 + (col >> 5)) * WR_FRAG, col & 31, y[m], b);
      }
    }
    __syncthreads();
  };
  phase_c();
  phase_f();
  // the first step's context: row 0 of the table; for a resumed window
  // context, from the refilled rings (nothing to wait for: those samples were
  // made before the launch); a call's step 0 has none
  if (table || (CTX && a.prev)) context(-1);
  publish(1u, cbv(bl0, 0), cbv(bl0 + 1, 0));
  const xw* YC = X + P.x_yc;
  const xw* YF = X + P.x_yf;
  for (int64_t t = 0; t + 1 < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    const float cb0 = cbv(bl0, t + 1), cb1 = cbv(bl0 + 1, t + 1);
    const bool tr = g == 0 && k == 0 && tid == 0;
    if (tr) trace_at(a, t, 16);
    if (ahead) {
      context(t);
      if (misc[0]) return;
    }
    gather_half(YC, tag, 0);
    if (misc[0]) return;
    if (tr) trace_at(a, t, 17);
    phase_c();
    if (tr) trace_at(a, t, 18);
    gather_half(YF, tag, KT);
    if (misc[0]) return;
    if (tr) trace_at(a, t, 19);
    phase_f();
    if (CTX && !ahead) {
      context(t);
      if (misc[0]) return;
    }
    publish(tag + 1, cb0, cb1);
    if (tr) trace_at(a, t, 20);
    if (g == 0 && k > 0 && k < 8 && tid == 0) trace_at(a, t, 24 + k);
  }
}

}  // namespace

template <int KH, bool CTX, int L, bool LAG, bool FL>
__global__ __launch_bounds__(WR_THREADS, 1) void wr_batch_kernel(BatchArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  int g = 0;
  const int r = wr_batch_role(a.P, blockIdx.x, &g);
  if (r < 0) return;
  if (r < a.P.NH) bhead_role<KH, CTX, L, LAG, FL>(a, g, r, lds);
  else bunit_role<KH, CTX, L, LAG, FL>(a, g, r - a.P.NH, lds);
}

template <int KH, int L>
static const void* batch_ptr_l(bool ctx, bool lag) {
  if (!ctx) return (const void*)wr_batch_kernel<KH, false, L, false, false>;
  return lag ? (const void*)wr_batch_kernel<KH, true, L, true, false>
             : (const void*)wr_batch_kernel<KH, true, L, false, false>;
}

// The synchronization floor of the batched launches (WaveRNN-896 and the
// smallest plan only).
template <int KH, int L>
static const void* floor_ptr_l(bool ctx, bool lag) {
  if (!ctx) return (const void*)wr_batch_kernel<KH, false, L, false, true>;
  return lag ? (const void*)wr_batch_kernel<KH, true, L, true, true>
             : (const void*)wr_batch_kernel<KH, true, L, false, true>;
}

const void* wr_batch_floor_kernel_ptr(int KH, bool ctx, int L, bool lag) {
  if (lag && !ctx) return nullptr;
  if (KH == 7) return L == 2 ? floor_ptr_l<7, 2>(ctx, lag) : L == 4 ? floor_ptr_l<7, 4>(ctx, lag)
                      : L == 8 ? floor_ptr_l<7, 8>(ctx, lag) : nullptr;
  if (KH == 1) return L == 2 ? floor_ptr_l<1, 2>(ctx, lag) : L == 4 ? floor_ptr_l<1, 4>(ctx, lag)
                      : L == 8 ? floor_ptr_l<1, 8>(ctx, lag) : nullptr;
  return nullptr;
}

template <int KH>
static const void* batch_ptr(bool ctx, int L, bool lag) {
  if (L == 2) return batch_ptr_l<KH, 2>(ctx, lag);
  if (L == 4) return batch_ptr_l<KH, 4>(ctx, lag);
  if (L == 8) return batch_ptr_l<KH, 8>(ctx, lag);
  return nullptr;
}

const void* wr_batch_kernel_ptr(int KH, bool ctx, int L, bool lag) {
  if (lag && !ctx) return nullptr;
  switch (KH) {
    case 1: return batch_ptr<1>(ctx, L, lag);
    case 2: return batch_ptr<2>(ctx, L, lag);
    case 3: return batch_ptr<3>(ctx, L, lag);
    case 7: return batch_ptr<7>(ctx, L, lag);
    default: return nullptr;
  }
}
