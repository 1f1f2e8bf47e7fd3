// Persistent multi-workgroup WaveRNN sampler (batch 1 per launch).
//
// The whole utterance runs inside one launch (Sec. 2.1): weights stay in VGPRs
// and LDS across the launch, and every step evaluates the GRU of Eq. 2, the
// coarse head, the coarse draw, the fine half, the fine head and the fine draw.
// Workgroups exchange vectors through tagged 32-bit words (the fp32 value with
// its lowest mantissa bit replaced by the parity of the producing step)
// instead of grid-wide barriers.
//
// A step, on the NH head workgroups (all on one XCD):
//   coarse gates of every unit (every head, identically, from pre-activations
//   the unit workgroups published for this step)
//   -> own 64 rows of O1, relu, own 64 columns of O2 -> 256 partial logits
//   --one exchange--> every head sums the NH partials, draws c_t
//   -> fine gates of every unit -> O3 rows, O4 columns -> partial logits
//   --one exchange--> sum, draw f_t.
// Meanwhile the NU unit workgroups receive y_c and y_f and compute R h for
// the next step (the paper's "gate" work), adding bias + conditioning; from
// y_f to the next step's pre-activations (two exchanges and R_f y_f) is the
// longest chain of a step at H = 896, longer than the fine half's exchange
// and draw it runs beside.
#include "wr_unit.h"

// The draw wave of a head (or mirror) gathers the partial logits of all NK
// slices alone: lane l reads classes 4 l .. 4 l + 3 of every slice with one
// 16-byte load (a wave's load covers whole cache lines) and sums slices
// [0, NHP), then [NHP, NK), then adds the two (the sums and order of the
// two-thread gather, so every head and mirror draws the same class); the
// logits stay in registers and no barrier separates gather and draw, while
// the other waves go on to the next gate terms (measured at H = 896: 4.94 us
// per step, against 5.13 with the two-thread gather and its barriers).
template <int NK>
__device__ __forceinline__ bool gather_partials(const PersistArgs& a, const xw* src, uint32_t tag, float4* z) {
  constexpr int NHP = (NK + 1) / 2;
  const int lane = threadIdx.x & 63;
  // first probe after 4 x 64 clocks (measured at H = 896 with the partials in
  // the leads' L2: 2 or 4 best, 6 1.6% slower, 0 or 1 6% slower)
  __builtin_amdgcn_s_sleep(4);
  const uint32_t bytes = (uint32_t)(NK * a.P.x_ps * 4), lo = 16u * lane, ps = (uint32_t)a.P.x_ps * 4u;
  xw4 w[NK];
  uint32_t pending = 0;
  {
    const __amdgpu_buffer_rsrc_t r = xrsrc(xopaque(src), bytes);
#pragma unroll
    for (int k = 0; k < NK; ++k) w[k] = xpeek4(r, k * ps + lo);
  }
#pragma unroll
  for (int k = 0; k < NK; ++k)
    if (!xok4(w[k], tag)) pending |= 1u << k;
  if (pending) {
    WaitBudget wb{wr_clock(), 0};
    while (pending) {
      if (!wait_ok(wb, a.err, a.limit, a.err)) {
        *z = float4{0.0f, 0.0f, 0.0f, 0.0f};   // a valid draw follows; the step is abandoned after it
        return false;
      }
      const __amdgpu_buffer_rsrc_t r = xrsrc(xopaque(src), bytes);
#pragma unroll
      for (int k = 0; k < NK; ++k)
        if (pending >> k & 1u) w[k] = xpeek4(r, k * ps + lo);
#pragma unroll
      for (int k = 0; k < NK; ++k)
        if ((pending >> k & 1u) && xok4(w[k], tag)) pending &= ~(1u << k);
    }
  }
  float4 s0 = {0.0f, 0.0f, 0.0f, 0.0f}, s1 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    float4& d = k < NHP ? s0 : s1;
    d.x += xval(w[k].x);
    d.y += xval(w[k].y);
    d.z += xval(w[k].z);
    d.w += xval(w[k].w);
  }
  z->x = s0.x + s1.x;
  z->y = s0.y + s1.y;
  z->z = s0.z + s1.z;
  z->w = s0.w + s1.w;
  return true;
}

// ------------------------------------------------------------------ head role
// A head owns a slice of HR = 16 RT rows of O1 / O3 (RT row tiles; the 8
// waves split them into RT row tiles x KC = 8 / RT column-tile chunks of KH
// tiles each) and the matching HR columns of O2 / O4 (class tiles 2w, 2w+1 of
// wave w).  NK = Hh / HR slices per half.  Without SPLIT head j holds slice j
// of both output MLPs; with SPLIT heads j < NK hold slice j of the coarse MLP
// (O1, O2) and heads NK + j slice j of the fine MLP (O3, O4), half the
// registers each.
// Every head draws both classes and evaluates the gates (Eq. 2) of the halves
// it serves (both without SPLIT).  The work that does not depend on
// the class being drawn (reading R h from the units, the I* terms of the known
// inputs) runs on waves 0-6 while wave 7 draws; the rest follows the draw.
//  GU = 1 (Hh <= 448): thread u < Hh owns coarse unit u and fine unit Hh + u,
//   its state in registers.
//  GU > 1 (wide): waves 0-6 prepare the pre-activations of units tid + 448 m
//   into LDS, then all 8 waves finish units tid + 512 m; the state stays in
//   LDS (registers are short with the larger O-layer slices).
// All 8 waves run the MFMA layers and gather the partial logits (two threads
// per class); the gate threads of this head's slice of units publish it for
// the unit workgroups.
// MR (mirrors, dense GU = 1 only): a coarse gate's pre-activation is the
// units' coarse-column word plus the mirrors' fine-column word, and the fine
// rows' words and the fine partial logits are double-buffered by step parity.
template <int KH, int RT, int GU, bool SPLIT, bool MR = false>
__device__ __forceinline__ void head_role(const PersistArgs& a, int j, unsigned char* lds) {
  constexpr int KC = 8 / RT;                       // column-tile chunks
  constexpr int KT = KH * KC;                      // column tiles per half
  constexpr int HR = 16 * RT;                      // rows per head
  constexpr int KO = HR / 32;                      // column tiles of the O2 / O4 slice
  constexpr int NK = 2 * KT / RT;                  // slices per half (Hh / HR)
  constexpr int NH = SPLIT ? 2 * NK : NK;          // heads
  constexpr int NHP = (NK + 1) / 2;                // partials per gathering thread
  constexpr int DW = 7;                            // the draw wave (no gate preparation)
  constexpr bool WIDE = GU > 1;
  constexpr int Hh = 32 * KT;
  static_assert(8 % RT == 0 && KO >= 1, "head shape");
  const PersistPlan& P = a.P;
  const int H = P.H;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const bool coarse = !SPLIT || j < NK;           // runs the coarse MLP slice
  const bool fine = !SPLIT || j >= NK;             // runs the fine MLP slice
  const int jk = SPLIT ? j % NK : j;               // slice index
  unsigned char* imc = lds;                        // y_c operand image [KT]
  unsigned char* imf = SPLIT ? lds : imc + KT * WR_FRAG;   // y_f operand image [KT] (SPLIT: one image)
  unsigned char* imo = imf + KT * WR_FRAG;         // relu(first layer) image [KO]
  float* op = (float*)(imo + KO * WR_FRAG);        // [KC][HR] first-layer partials
  float* zs2 = op + KC * HR;                       // [256] sums over the second half of the heads
  float* zs = zs2 + 256;                           // [256] sums over the first half of the heads
  float* zk = zs + 256;                            // [256] logits of the last draw
  float* yv = zk + 256;                            // [Hh] (GU = 1) this half of h; (wide) h_c
  float* hfv = yv + Hh;                            // wide: [Hh] h_f
  float* pre = hfv + Hh;                           // wide: [5][Hh] prepared gate terms
  float* prf = pre + 5 * Hh;                       // wide: [4][Hh] fine words (u, r, e) and conditioning
  float* iws = prf + 4 * Hh;                       // wide: [Hh][15] I* of coarse (2) and fine (3) columns
  int* misc = (int*)(WIDE ? iws + 15 * Hh : yv + Hh);   // [0] abort [1] c_t [2] c_prev [3] f_prev
  float* fmisc = (float*)(misc + 8);               // [2] lse_c [3] z_c[c]
  float2* uni = (float2*)(misc + 16);              // [2][64] (u_c, u_f) of a batch of 64 steps
  int* tgt = (int*)(uni + 128);                    // [2][64] teacher-forcing targets of the batch

  // --- prologue: zero the operand images, load this wave's fragments
  for (int i = tid; i < ((SPLIT ? 1 : 2) * KT + KO) * WR_FRAG / 16; i += WR_THREADS) ((uint4*)lds)[i] = uint4{0, 0, 0, 0};
  // fragments: W1 [KH], W2 [2 KO] of the head's (first) MLP slice, then
  // without SPLIT W3 [KH], W4 [2 KO] of its fine slice; SPLIT: a fine head's
  // W1, W2 hold O3, O4
  constexpr int KH3 = SPLIT ? 1 : KH, KO4 = SPLIT ? 1 : 2 * KO;
  bf16x8 W1[KH], W3[KH3], W2[2 * KO], W4[KO4];
  {
    const uint4* src = a.hw + ((size_t)(j * 8 + wave) * P.hw_frags) * 64 + lane;
#pragma unroll
    for (int i = 0; i < KH; ++i) W1[i] = __builtin_bit_cast(bf16x8, src[(size_t)i * 64]);
    if (!SPLIT) {
#pragma unroll
      for (int i = 0; i < KH3; ++i) W3[i] = __builtin_bit_cast(bf16x8, src[(size_t)(KH + i) * 64]);
    }
    const uint4* s2 = src + (size_t)(SPLIT ? KH : 2 * KH) * 64;
#pragma unroll
    for (int i = 0; i < 2 * KO; ++i) W2[i] = __builtin_bit_cast(bf16x8, s2[(size_t)i * 64]);
    if (!SPLIT) {
#pragma unroll
      for (int i = 0; i < KO4; ++i) W4[i] = __builtin_bit_cast(bf16x8, s2[(size_t)(2 * KO + i) * 64]);
    }
  }
  // GU = 1: gate thread u < Hh.  I* coefficients: coarse row (c_{t-1}, f_{t-1}),
  // fine row (c_{t-1}, f_{t-1}, c_t) of each gate.
  const bool gate = tid < Hh;
  const int u = tid;
  float ic[3][2], ifn[3][3];
  float hc = 0.0f, hf = 0.0f;
  if (!WIDE && gate) {
#pragma unroll
    for (int g = 0; g < 3; ++g) {
      ic[g][0] = a.Iw[3 * (g * H + u) + 0];
      ic[g][1] = a.Iw[3 * (g * H + u) + 1];
      ifn[g][0] = a.Iw[3 * (g * H + Hh + u) + 0];
      ifn[g][1] = a.Iw[3 * (g * H + Hh + u) + 1];
      ifn[g][2] = a.Iw[3 * (g * H + Hh + u) + 2];
    }
    if (a.h_in) {
      hc = a.h_in[u];
      hf = a.h_in[Hh + u];
    }
  }
  if (WIDE) {
    for (int v = tid; v < Hh; v += WR_THREADS) {
#pragma unroll
      for (int g = 0; g < 3; ++g) {
        iws[15 * v + 5 * g + 0] = a.Iw[3 * (g * H + v) + 0];
        iws[15 * v + 5 * g + 1] = a.Iw[3 * (g * H + v) + 1];
        iws[15 * v + 5 * g + 2] = a.Iw[3 * (g * H + Hh + v) + 0];
        iws[15 * v + 5 * g + 3] = a.Iw[3 * (g * H + Hh + v) + 1];
        iws[15 * v + 5 * g + 4] = a.Iw[3 * (g * H + Hh + v) + 2];
      }
      yv[v] = a.h_in ? a.h_in[v] : 0.0f;
      hfv[v] = a.h_in ? a.h_in[Hh + v] : 0.0f;
    }
  }
  const float b1r = tid < HR && coarse ? a.b1[jk * HR + tid] : 0.0f;
  const float b3r = tid < HR && fine ? a.b3[jk * HR + tid] : 0.0f;
  const float4 b2l = wave == DW ? *(const float4*)(a.b2 + 4 * lane) : float4{0, 0, 0, 0};
  const float4 b4l = wave == DW ? *(const float4*)(a.b4 + 4 * lane) : float4{0, 0, 0, 0};
  if (tid == 0) {
    misc[0] = 0;
    misc[2] = a.c_in ? a.c_in[0] : 128;
    misc[3] = a.f_in ? a.f_in[0] : 0;
  }
  const xw* GA = a.xc + P.x_ga;
  const xw* GF = a.xc + P.x_gf;
  xw* YC = a.xc + P.x_yc;
  xw* YF = a.xc + P.x_yf;
  xw* PCo = a.xc + P.x_pc + (size_t)jk * P.x_ps;
  xw* PFo = a.xc + P.x_pf + (size_t)jk * P.x_ps;
  const xw* HF = a.xc + P.x_hf;
  const xw* PC = a.xc + P.x_pc;
  const xw* PF = a.xc + P.x_pf;
  const int rt = wave % RT, kc = wave / RT;        // first layer: row tile, column-tile chunk
  // GU = 1: pre-activation words of this thread's units, loaded ahead (MR:
  // the units' three, then the mirrors' three of the coarse half)
  constexpr int NCW = MR ? 6 : 3;
  xw pc[NCW] = {}, pf[3] = {0, 0, 0};
  float cbe_c = 0.0f, cbe_f = 0.0f;
  auto prefetch_coarse = [&](int64_t n) {
    if (!WIDE && gate && coarse) {
      pc[0] = xpeek(GA + u); pc[1] = xpeek(GA + Hh + u); pc[2] = xpeek(GA + 2 * Hh + u);
      if (MR) { pc[3] = xpeek(HF + u); pc[4] = xpeek(HF + Hh + u); pc[5] = xpeek(HF + 2 * Hh + u); }
      cbe_c = cb_row(a, n)[2 * H + u];
    }
  };
  // the fine rows' words of launch step t (its buffer with MR)
  auto prefetch_fine = [&](int64_t t) {
    if (!WIDE && gate && fine) {
      const xw* G = GF + wr_dbuf(t, P.x_gfs);
      pf[0] = xpeek(G + u); pf[1] = xpeek(G + Hh + u); pf[2] = xpeek(G + 2 * Hh + u);
      cbe_f = cb_row(a, a.t0 + t)[2 * H + Hh + u];
    }
  };
  // first layer on the 8 waves -> relu -> operand image of the second layer
  auto first_layer = [&](const bf16x8* W, const unsigned char* img, float b) {
    f32x4 acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < KH; i += 2) {
      acc0 = mfma(afrag(img, kc * KH + i), W[i], acc0);
      if (i + 1 < KH) acc1 = mfma(afrag(img, kc * KH + i + 1), W[i + 1], acc1);
    }
    if (lane < 16) op[kc * HR + 16 * rt + lane] = mfma_row(acc0) + mfma_row(acc1);
    __syncthreads();
    if (tid < HR) {
      float s = op[tid];
#pragma unroll
      for (int q = 1; q < KC; ++q) s += op[q * HR + tid];
      aput(imo + (tid >> 5) * WR_FRAG, tid & 31, wr_relu(s + b));
    }
    __syncthreads();
  };
  // second layer: class tiles 2*wave, 2*wave+1 over this head's HR columns
  bool lx = false;   // heads (and mirrors) share one XCD (leads_share_xcd)
  auto second_layer = [&](const bf16x8* W, xw* dst, uint32_t tag) {
    f32x4 A = {0, 0, 0, 0}, B = {0, 0, 0, 0};
#pragma unroll
    for (int kt = 0; kt < KO; ++kt) {
      const bf16x8 x = afrag(imo, kt);
      A = mfma(x, W[kt], A);
      B = mfma(x, W[KO + kt], B);
    }
    if (lane < 16) {
      xpub_l(dst + 32 * wave + lane, tag, mfma_row(A), lx);
      xpub_l(dst + 32 * wave + 16 + lane, tag, mfma_row(B), lx);
    }
  };
  // partial logits of all slices: thread (v, half) sums its half of the
  // slices in slice order, each word checked for its tag.  The partials are
  // being published as this head starts to wait, so the first probe waits a
  // little (a probe at once comes back without them, and every failed probe
  // of the whole grid loads the exchange; measured: 7 slices 5.17 us per
  // step with a 6 x 64-clock delay, 5.59 without, 5.64 with the flag phase
  // below).  With split heads (16 slices, 8 words per thread) lane jj of
  // every wave first waits for the last word of slice jj, so that while the
  // exchange is in flight only those words are polled.
  auto gather_logits = [&](const xw* src, uint32_t tag) {
    if (SPLIT) __builtin_amdgcn_s_sleep(12);
    else __builtin_amdgcn_s_sleep(6);
    if (SPLIT) {   // every wave waits on the flags itself: no barrier before the reads
      float y;
      const int jj = lane < NK ? lane : 0;
      if (!poll_sleepy<false>(src + (size_t)jj * P.x_ps + 255, tag, &y, a)) misc[0] = 1;
    }
    float s;
    const int v = tid & 255, hh = tid >> 8;
    if (!sum_parts<NHP>(src, P.x_ps, hh ? NHP : 0, hh ? NK : NHP, v, tag, &s, a)) misc[0] = 1;
    else (hh ? zs2 : zs)[v] = s;
  };
  auto gather_wave = [&](const xw* src, uint32_t tag, float4* z) -> bool {
    return gather_partials<NK>(a, src, tag, z);
  };
  // Philox blocks of steps t .. t+63 into batch buffer b, one step per lane of
  // the draw wave: the 64-bit multiplies cost the same for 64 lanes as for one
  auto fill_batch = [&](int64_t t, int b) {
    const int64_t s = t + lane;
    if (s < a.T) {
      float uc, uf;
      wr_uniforms(a.seed, a.stream_id, (uint64_t)(a.t0 + s), &uc, &uf);
      uni[b * 64 + lane] = float2{uc, uf};
      tgt[b * 64 + lane] = a.target ? a.target[s] : 0;
    }
  };
  if (wave == DW) fill_batch(0, 0);
  __syncthreads();
  prefetch_coarse(a.t0);
  prefetch_fine(0);
  const bool trw = j == 0 && tid == WR_THREADS - 64;       // tracing thread (draw wave)
  // wide: the units publish a step's coarse and fine words together, so both
  // are read at once (one round trip) with the conditioning of the e gates:
  // coarse terms into pre, the fine words and conditioning into prf
  // Word k of a thread: half k / (3 GU) (GA, GF), slot m = k / 3 % GU, gate
  // k % 3; its value lands in LDS (pre rows 0-2 or prf rows 0-2) as it arrives.
  auto wide_words = [&](uint32_t tag, float x0, int64_t n) -> bool {
    if (wave == DW) return true;
    constexpr int NW = 6 * GU;
    const float* cbr = cb_row(a, n) + 2 * H;
    int un[GU];
    float cbc[GU], cbf[GU];
#pragma unroll
    for (int m = 0; m < GU; ++m) {
      un[m] = tid + 448 * m < Hh ? tid + 448 * m : tid;
      cbc[m] = cbr[un[m]];
      cbf[m] = cbr[Hh + un[m]];
    }
    // with split MLPs a head reads only the half it evaluates
    uint32_t pending = (coarse ? (1u << 3 * GU) - 1 : 0u) | (fine ? ((1u << 3 * GU) - 1) << 3 * GU : 0u);
    WaitBudget wb{wr_clock(), 0};
    for (;;) {
      xw x[NW];
#pragma unroll
      for (int k = 0; k < NW; ++k)
        x[k] = (pending >> k & 1u) ? xpeek((k < 3 * GU ? GA : GF) + (k % 3) * Hh + un[k / 3 % GU]) : 0;
#pragma unroll
      for (int k = 0; k < NW; ++k)
        if ((pending >> k & 1u) && xok(x[k], tag)) {
          (k < 3 * GU ? pre : prf)[(k % 3) * Hh + un[k / 3 % GU]] = xval(x[k]);
          pending &= ~(1u << k);
        }
      if (!pending) break;
      if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
    }
#pragma unroll
    for (int m = 0; m < GU; ++m) {
      if (tid + 448 * m >= Hh) continue;
      const int v = un[m];
      const float* iv = iws + 15 * v;
      pre[v] = pre[v] + iv[0] * x0;
      pre[Hh + v] = pre[Hh + v] + iv[5] * x0;
      pre[3 * Hh + v] = iv[10] * x0;
      pre[4 * Hh + v] = cbc[m];
      prf[3 * Hh + v] = cbf[m];
    }
    return true;
  };
  float cu = 0.0f, cr = 0.0f, ce = 0.0f, cie = 0.0f;       // GU = 1, coarse: before f_{t-1} is known
  float fu = 0.0f, fr = 0.0f, fe = 0.0f, fie = 0.0f;       // GU = 1, fine: before c_t is known
  // coarse gate terms known before f_{t-1} (n: the step's sample index)
  auto coarse_pre = [&](uint32_t tag, float x0, int64_t n) {
    if (WIDE) {
      if (!wide_words(tag, x0, n)) misc[0] = 1;
      return;
    }
    if (!gate || !coarse) return;
    // the units publish these words at about the time this head starts to
    // wait for them, so the first probe goes out a little later (measured at
    // H = 896: 5.12 us per step, against 5.22 with the probe issued at the
    // end of the fine gather).  With mirrors, whose words stay in the leads'
    // L2, 5 x 64 clocks (3 to 5 best, 8 1.4% slower, 0 or 1 5% slower)
    __builtin_amdgcn_s_sleep(MR ? 5 : 8);
    prefetch_coarse(n);
    const xw* ps[6] = {GA + u, GA + Hh + u, GA + 2 * Hh + u, HF + u, HF + Hh + u, HF + 2 * Hh + u};
    float v[NCW];
    if (!poll_pref<NCW>(ps, pc, tag, v, a)) {
      misc[0] = 1;
      return;
    }
    if (MR) {   // the units' coarse-column part plus the mirrors' fine-column part
      v[0] = v[0] + v[3];
      v[1] = v[1] + v[4];
      v[2] = v[2] + v[5];
    }
    cu = v[0] + ic[0][0] * x0;
    cr = v[1] + ic[1][0] * x0;
    ce = v[2];
    cie = ic[2][0] * x0;
  };
  auto fine_pre = [&](int64_t t, float x0, float x1) {
    if (WIDE) {   // from the words read with the coarse ones (LDS only)
      if (!fine) return;
      for (int un = tid; un < Hh; un += 448) {
        const float* iv = iws + 15 * un;
        pre[un] = prf[un] + __builtin_fmaf(iv[3], x1, iv[2] * x0);
        pre[Hh + un] = prf[Hh + un] + __builtin_fmaf(iv[8], x1, iv[7] * x0);
        pre[2 * Hh + un] = prf[2 * Hh + un];
        pre[3 * Hh + un] = __builtin_fmaf(iv[13], x1, iv[12] * x0);
        pre[4 * Hh + un] = prf[3 * Hh + un];
      }
      return;
    }
    if (!gate || !fine) return;
    const xw* G = GF + wr_dbuf(t, P.x_gfs);
    const xw* ps[3] = {G + u, G + Hh + u, G + 2 * Hh + u};
    float v[3];
    if (!poll_pref<3>(ps, pf, wr_dtag(t, P.x_gfs), v, a)) {
      misc[0] = 1;
      return;
    }
    fu = v[0] + __builtin_fmaf(ifn[0][1], x1, ifn[0][0] * x0);
    fr = v[1] + __builtin_fmaf(ifn[1][1], x1, ifn[1][0] * x0);
    fe = v[2];
    fie = __builtin_fmaf(ifn[2][1], x1, ifn[2][0] * x0);
  };
  // wide: finish the gates of units tid + 512 m with the drawn input x (I*
  // column q of the row) into h (LDS) and the operand image
  auto wide_gates = [&](float x, int q, float* h, unsigned char* img, xw* Y, uint32_t tag) {
#pragma unroll
    for (int m = 0; m < (Hh + WR_THREADS - 1) / WR_THREADS; ++m) {
      const int un = tid + WR_THREADS * m;
      if (un >= Hh) break;
      const float* iv = iws + 15 * un;
      const float uu = fsig(__builtin_fmaf(iv[q], x, pre[un]));
      const float rr = fsig(__builtin_fmaf(iv[5 + q], x, pre[Hh + un]));
      const float e = ftanh(__builtin_fmaf(rr, pre[2 * Hh + un], __builtin_fmaf(iv[10 + q], x, pre[3 * Hh + un]) + pre[4 * Hh + un]));
      const float hn = __builtin_fmaf(uu, h[un], (1.0f - uu) * e);
      h[un] = hn;
      aput(img + (un >> 5) * WR_FRAG, un & 31, hn);
      if ((unsigned)(un - HR * jk) < (unsigned)HR) xpub(Y + un, tag, hn);   // this head's slice, for the units
    }
  };
  // before step 0's coarse gates, which wait for the mirrors' first words:
  // the mirrors check the XCDs before they publish those
  if (WR_LOCAL_XCHG && P.x_xcc) lx = leads_share_xcd(a.xc + P.x_xcc, P.NH + P.NM, j, misc + 4, a);
  coarse_pre(1u, fscale(misc[2]), a.t0);
  // Every prologue load has landed: no wait inside the loop is left waiting on
  // them (a wait there would also wait for the wave's outstanding stores).
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (misc[0]) return;

  for (int64_t t = 0; t < a.T; ++t) {
    const int64_t n = a.t0 + t;
    const uint32_t tag = (uint32_t)(t + 1);
    if (trw) trace_at(a, t, 0);
    const int bs = (int)((t >> 6) & 1) * 64 + (int)(t & 63);   // this step in the batch buffers
    if (wave == DW && (t & 63) == 0) fill_batch(t + 64, (int)(((t >> 6) + 1) & 1));
    // (1) coarse gates of every unit, finished with f_{t-1}
    if (WIDE) {
      if (coarse) wide_gates(fscale(misc[3]), 1, yv, imc, YC, tag);
    } else if (gate && coarse) {
      const float x1 = fscale(misc[3]);
      const float uu = fsig(__builtin_fmaf(ic[0][1], x1, cu)), rr = fsig(__builtin_fmaf(ic[1][1], x1, cr));
      const float e = ftanh(__builtin_fmaf(rr, ce, __builtin_fmaf(ic[2][1], x1, cie) + cbe_c));
      hc = __builtin_fmaf(uu, hc, (1.0f - uu) * e);
      aput(imc + (u >> 5) * WR_FRAG, u & 31, hc);
      yv[u] = hc;
      if (u - HR * jk < (unsigned)HR) xpub(YC + u, tag, hc);   // this head's slice, for the units
    }
    __syncthreads();
    if (trw) trace_at(a, t, 1);
    if (trw) trace_at(a, t, 19);
    // (2) own rows of O1 -> relu -> own columns of O2 -> partial coarse logits
    if (coarse) {
      first_layer(W1, imc, b1r);
      if (trw) trace_at(a, t, 2);
      second_layer(W2, PCo, tag);
      if (trw) trace_at(a, t, 3);
    }
    if (j == NH - 1 && tid == WR_THREADS - 64) trace_at(a, t, 13);
    if (j > 0 && j < 8 && tid == WR_THREADS - 64) trace_at(a, t, 24 + j);
    // (3) coarse logits of all heads; this step's fine words are loaded
    if (SPLIT) {
      gather_logits(PC, tag);
      if (trw) trace_at(a, t, 15);
    }
    if (t > 0) prefetch_fine(t);
    if (SPLIT) {
      __syncthreads();
      if (misc[0]) return;
      if (trw) trace_at(a, t, 4);
    }
    // (4) draw c_t on the draw wave; meanwhile the fine gates start
    if (wave == DW) {
      float lse;
      const int forced = a.target ? (tgt[bs] >> 8) : -1;
      int c = 0;
      if (SPLIT) {
        c = draw_wave(zs, zs2, b2l, uni[bs].x, forced, zk, a.nll_out ? &lse : nullptr);
      } else {
        float4 z;
        if (!gather_wave(PC, tag, &z)) misc[0] = 1;
        if (trw) trace_at(a, t, 15);
        c = draw_z(z, b2l, uni[bs].x, forced, zk, a.nll_out ? &lse : nullptr);
      }
      if (trw) trace_at(a, t, 16);
      if (j == 0 && a.zc_out) *(float4*)(a.zc_out + t * WR_CLASSES + 4 * lane) = *(const float4*)(zk + 4 * lane);
      if (lane == 0) {
        misc[1] = c;
        if (a.nll_out) {
          fmisc[2] = lse;
          fmisc[3] = zk[c];
        }
      }
    } else {
      fine_pre(t, fscale(misc[2]), fscale(misc[3]));
    }
    __syncthreads();
    if (misc[0]) return;
    if (trw) trace_at(a, t, 5);
    // (5) fine gates of every unit, finished with c_t (c_t reaches the fine half only)
    const int c = misc[1];
    if (WIDE) {
      if (fine) wide_gates(fscale(c), 4, hfv, imf, YF, tag);
    } else if (gate && fine) {
      const float x2 = fscale(c);
      const float uu = fsig(__builtin_fmaf(ifn[0][2], x2, fu)), rr = fsig(__builtin_fmaf(ifn[1][2], x2, fr));
      const float e = ftanh(__builtin_fmaf(rr, fe, __builtin_fmaf(ifn[2][2], x2, fie) + cbe_f));
      hf = __builtin_fmaf(uu, hf, (1.0f - uu) * e);
      aput(imf + (u >> 5) * WR_FRAG, u & 31, hf);
      yv[u] = hf;
      if (u - HR * jk < (unsigned)HR) xpub(YF + u, tag, hf);
    }
    __syncthreads();
    if (trw) trace_at(a, t, 6);
    if (trw) trace_at(a, t, 22);
    // (6) own rows of O3 -> relu -> own columns of O4 -> partial fine logits
    if (fine) {
      if (SPLIT) {
        first_layer(W1, imf, b3r);
        second_layer(W2, PFo + wr_dbuf(t, P.x_pfs), wr_dtag(t, P.x_pfs));
      } else {
        first_layer(W3, imf, b3r);
        if (trw) trace_at(a, t, 7);
        second_layer(W4, PFo + wr_dbuf(t, P.x_pfs), wr_dtag(t, P.x_pfs));
        if (trw) trace_at(a, t, 8);
      }
    }
    if (j == NH - 1 && tid == WR_THREADS - 64) trace_at(a, t, 14);
    // (7) fine logits of all heads
    if (SPLIT) {
      gather_logits(PF + wr_dbuf(t, P.x_pfs), wr_dtag(t, P.x_pfs));
      if (trw) trace_at(a, t, 17);
      __syncthreads();
      if (misc[0]) return;
      if (trw) trace_at(a, t, 9);
    }
    // (8) draw f_t on the draw wave; meanwhile the next coarse gates start
    if (wave == DW) {
      float lse;
      const int forced = a.target ? (tgt[bs] & 255) : -1;
      int f = 0;
      if (SPLIT) {
        f = draw_wave(zs, zs2, b4l, uni[bs].y, forced, zk, a.nll_out ? &lse : nullptr);
      } else {
        float4 z;
        if (!gather_wave(PF + wr_dbuf(t, P.x_pfs), wr_dtag(t, P.x_pfs), &z)) misc[0] = 1;
        if (trw) trace_at(a, t, 17);
        f = draw_z(z, b4l, uni[bs].y, forced, zk, a.nll_out ? &lse : nullptr);
      }
      if (trw) trace_at(a, t, 18);
      if (j == 0 && a.zf_out) *(float4*)(a.zf_out + t * WR_CLASSES + 4 * lane) = *(const float4*)(zk + 4 * lane);
      if (lane == 0) {
        if (j == 0) {
          if (a.out) a.out[t] = (uint16_t)(256 * c + f);
          if (a.nll_out) a.nll_out[t] = (fmisc[2] - fmisc[3]) + (lse - zk[f]);
        }
        misc[2] = c;
        misc[3] = f;
      }
    } else if (t + 1 < a.T) {
      coarse_pre(tag + 1, fscale(c), n + 1);
    }
    __syncthreads();
    if (misc[0]) return;
    if (trw) trace_at(a, t, 10);
  }
  // final state: head 0 writes the halves it evaluated, head NK the fine half with split MLPs
  if (a.h_out && (j == 0 || (SPLIT && j == NK))) {
    if (WIDE) {
      for (int v = tid; v < Hh; v += WR_THREADS) {
        if (coarse) a.h_out[v] = yv[v];
        if (fine) a.h_out[Hh + v] = hfv[v];
      }
    } else if (gate) {
      if (coarse) a.h_out[u] = hc;
      if (fine) a.h_out[Hh + u] = hf;
    }
  }
  if (j == 0) {
    if (tid == 0) {
      if (a.c_out) a.c_out[0] = (uint8_t)misc[2];
      if (a.f_out) a.f_out[0] = (uint8_t)misc[3];
    }
  }
}

// ------------------------------------------------------------------ mirror role
// Mirror j draws c_t as every head does (the same partial logits summed in
// the same order, the same uniform or target), evaluates the fine gates of
// every unit (Eq. 2, with c_t) with a head's arithmetic, and forms the
// products of the coarse rows with the new y_f for the next step: coarse row
// tiles 12 j .. 12 j + 11 over the fine columns (wave w: row tiles
// 3 (w % 4) .. +2 over the column tiles of half w / 4, the halves added in
// LDS).  The heads add them to the units' coarse-column words.  y_f enters
// the products as the exchange delivers values (lowest bit cleared), so the
// teacher-forced scoring recurrence forms the same sums.  The mirror then
// draws f_t as the heads do, for the next step's input terms.
// Exchange order: the words of step t + 1 are published after c_t, and a head
// publishes the partials of c_{t+1} only after reading them, so one buffer
// holds them.  A mirror reads the fine partials of step t after publishing
// those words: a head publishes fine partials of step t + 2 only after the
// mirrors' words of step t + 2, which follow f_t, so two buffers by step
// parity suffice; the fine rows' words likewise.
template <int KH>
__device__ __forceinline__ void mirror_role(const PersistArgs& a, int j, unsigned char* lds) {
  constexpr int KT = 2 * KH;                       // column tiles per half
  constexpr int MK = KT / 2;                       // column tiles per wave (half of the fine columns)
  constexpr int NK = KH;                           // slices of the partial logits (Hh / 64 heads)
  constexpr int DW = 7;                            // the draw wave
  constexpr int Hh = 32 * KT;
  constexpr int MRW = 16 * WR_MTILES;              // rows of a mirror
  const PersistPlan& P = a.P;
  const int H = P.H;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  unsigned char* imf = lds;                        // [KT] operand image of y_f
  float* part = (float*)(imf + KT * WR_FRAG);      // [2][MRW] products of the two column halves
  float* zk = part + 2 * MRW;                      // [256] logits of the last draw
  int* misc = (int*)(zk + 256);                    // [0] abort [1] c_t [2] c_prev [3] f_prev
  float2* uni = (float2*)(misc + 16);              // [2][64] (u_c, u_f) of a batch of 64 steps
  int* tgt = (int*)(uni + 128);                    // [2][64] teacher-forcing targets of the batch
  for (int i = tid; i < KT * WR_FRAG / 16; i += WR_THREADS) ((uint4*)imf)[i] = uint4{0, 0, 0, 0};
  const int rq = wave & 3, kh = wave >> 2;         // row tiles 3 rq .. 3 rq + 2, column half kh
  bf16x8 W[3 * MK];
  {
    const uint4* src = a.mw + ((size_t)(j * 8 + wave) * P.mw_frags) * 64 + lane;
#pragma unroll
    for (int i = 0; i < 3 * MK; ++i) W[i] = __builtin_bit_cast(bf16x8, src[(size_t)i * 64]);
  }
  // gate thread u < Hh: fine unit Hh + u, its I* coefficients (c_{t-1}, f_{t-1}, c_t) and state
  const bool gate = tid < Hh;
  const int u = tid;
  float ifn[3][3];
  float hf = 0.0f;
  if (gate) {
#pragma unroll
    for (int g = 0; g < 3; ++g)
#pragma unroll
      for (int q = 0; q < 3; ++q) ifn[g][q] = a.Iw[3 * (g * H + Hh + u) + q];
    if (a.h_in) hf = a.h_in[Hh + u];
  }
  const float4 b2l = wave == DW ? *(const float4*)(a.b2 + 4 * lane) : float4{0, 0, 0, 0};
  const float4 b4l = wave == DW ? *(const float4*)(a.b4 + 4 * lane) : float4{0, 0, 0, 0};
  if (tid == 0) {
    misc[0] = 0;
    misc[2] = a.c_in ? a.c_in[0] : 128;
    misc[3] = a.f_in ? a.f_in[0] : 0;
  }
  const xw* GF = a.xc + P.x_gf;
  const xw* PC = a.xc + P.x_pc;
  const xw* PF = a.xc + P.x_pf;
  xw* HF = a.xc + P.x_hf + (size_t)MRW * j;
  // Philox blocks of steps t .. t+63 into batch buffer b (as the heads draw them)
  auto fill_batch = [&](int64_t t, int b) {
    const int64_t s = t + lane;
    if (s < a.T) {
      float uc, uf;
      wr_uniforms(a.seed, a.stream_id, (uint64_t)(a.t0 + s), &uc, &uf);
      uni[b * 64 + lane] = float2{uc, uf};
      tgt[b * 64 + lane] = a.target ? a.target[s] : 0;
    }
  };
  if (wave == DW) fill_batch(0, 0);
  __syncthreads();
  if (gate) aput(imf + (u >> 5) * WR_FRAG, u & 31, xround(hf));
  bool lx = false;   // heads and mirrors share one XCD (leads_share_xcd)
  // the coarse rows' products with y_f for step s, published for the heads
  auto products = [&](int64_t s) {
    f32x4 acc[3];
#pragma unroll
    for (int r = 0; r < 3; ++r) acc[r] = f32x4{0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < MK; ++i) {
      const bf16x8 x = afrag(imf, kh * MK + i);
#pragma unroll
      for (int r = 0; r < 3; ++r) acc[r] = mfma(x, W[r * MK + i], acc[r]);
    }
    if (lane < 16) {
#pragma unroll
      for (int r = 0; r < 3; ++r) part[kh * MRW + 16 * (3 * rq + r) + lane] = mfma_row(acc[r]);
    }
    __syncthreads();
    if (tid < MRW) xpub_l(HF + tid, (uint32_t)s + 1u, part[tid] + part[MRW + tid], lx);
  };
  __builtin_amdgcn_s_waitcnt(0);   // prologue loads in before the loop (see head_role)
  __syncthreads();
  if (WR_LOCAL_XCHG) lx = leads_share_xcd(a.xc + P.x_xcc, P.NH + P.NM, P.NH + j, misc + 4, a);
  products(0);
  float fu = 0.0f, fr = 0.0f, fe = 0.0f, fie = 0.0f, cbe = 0.0f;
  for (int64_t t = 0; t < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    const int bs = (int)((t >> 6) & 1) * 64 + (int)(t & 63);
    if (wave == DW && (t & 63) == 0) fill_batch(t + 64, (int)(((t >> 6) + 1) & 1));
    // (1) c_t on the draw wave; the fine rows' words of step t on the gate threads
    if (wave == DW) {
      float4 z;
      if (!gather_partials<NK>(a, PC, tag, &z)) misc[0] = 1;
      const int c = draw_z(z, b2l, uni[bs].x, a.target ? (tgt[bs] >> 8) : -1, zk, nullptr);
      if (lane == 0) misc[1] = c;
    } else if (gate) {
      const xw* G = GF + wr_dbuf(t, P.x_gfs);
      const xw* ps[3] = {G + u, G + Hh + u, G + 2 * Hh + u};
      const xw w0[3] = {xpeek(ps[0]), xpeek(ps[1]), xpeek(ps[2])};
      cbe = cb_row(a, a.t0 + t)[2 * H + Hh + u];
      float v[3];
      if (!poll_pref<3>(ps, w0, wr_dtag(t, P.x_gfs), v, a)) {
        misc[0] = 1;
      } else {
        const float x0 = fscale(misc[2]), x1 = fscale(misc[3]);
        fu = v[0] + __builtin_fmaf(ifn[0][1], x1, ifn[0][0] * x0);
        fr = v[1] + __builtin_fmaf(ifn[1][1], x1, ifn[1][0] * x0);
        fe = v[2];
        fie = __builtin_fmaf(ifn[2][1], x1, ifn[2][0] * x0);
      }
    }
    __syncthreads();
    if (misc[0]) return;
    // (2) the fine gates with c_t, as a head evaluates them
    if (gate) {
      const float x2 = fscale(misc[1]);
      const float uu = fsig(__builtin_fmaf(ifn[0][2], x2, fu)), rr = fsig(__builtin_fmaf(ifn[1][2], x2, fr));
      const float e = ftanh(__builtin_fmaf(rr, fe, __builtin_fmaf(ifn[2][2], x2, fie) + cbe));
      hf = __builtin_fmaf(uu, hf, (1.0f - uu) * e);
      aput(imf + (u >> 5) * WR_FRAG, u & 31, xround(hf));
    }
    __syncthreads();
    // (3) the coarse rows' products with y_f for step t + 1
    if (t + 1 < a.T) products(t + 1);
    if (j == 0 && tid == 0) trace_at(a, t, 23);
    // (4) f_t on the draw wave
    if (wave == DW) {
      float4 z;
      if (!gather_partials<NK>(a, PF + wr_dbuf(t, P.x_pfs), wr_dtag(t, P.x_pfs), &z)) misc[0] = 1;
      const int f = draw_z(z, b4l, uni[bs].y, a.target ? (tgt[bs] & 255) : -1, zk, nullptr);
      if (lane == 0) {
        misc[2] = misc[1];
        misc[3] = f;
      }
    }
    __syncthreads();
    if (misc[0]) return;
  }
}

template <int KH>
__global__ __launch_bounds__(WR_THREADS, 1) void wr_persist_kernel(PersistArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int r = wr_role(a.P, blockIdx.x);
  if (r < 0) return;
  if (r < a.P.NH) head_role<KH, 4, 1, false, true>(a, r, lds);
  else if (r < a.P.NH + a.P.NM) mirror_role<KH>(a, r - a.P.NH, lds);
  else unit_role<KH, false, true>(a, r - a.P.NH - a.P.NM, lds);
}

// ------------------------------------------------------------ block-sparse unit role
// Unit k of a block-sparse R (Sec. 3.2): rows SR k .. SR k + SR - 1 of the
// stacked gate matrices, SL lanes of waves 0-3 per row, each walking its part
// of its block-row's kept blocks (layout in sparse_plan) against h in LDS:
// per 4 x 4 block one shared column index, the row's 4 weights and 4
// consecutive h values (one 16-byte read); per 16 x 1 block the index, one
// weight and one h value that all 16 rows of the block read (four blocks'
// weights and indices per read); waves 4-7 gather h.
__device__ __forceinline__ void sparse_unit_role(const PersistArgs& a, int k, unsigned char* lds) {
  const PersistPlan& P = a.P;
  const int H = P.H, Hh = P.Hh, SL = P.SL, NRC = P.NRC, NRF = P.NRF, BR = P.BR;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const unsigned char* wts = lds;                           // [NRC + NRF][256] block rows of weights
  const uint16_t* bix = (const uint16_t*)(lds + P.u_wb);    // [NRC + NRF][BR][SL] block-column indices
  float* hv = (float*)(lds + P.u_lds_w);          // [H] h of the last step
  int* misc = (int*)(hv + H);
  const bool cw = tid < 256;                      // computing (and publishing) lanes
  const int ru = (tid & 255) / SL, part = tid % SL;   // row in the unit, part of its block-row's blocks
  const int row = P.SR * k + ru;                  // R row g H + i of a computing lane
  const int bro = ru / P.BH;                      // block-row in the unit
  const bool lead = cw && tid % SL == 0;
  const int g = row / H, i = row % H;
  const bool fine = i >= Hh;
  xw* dst = a.xc + (fine ? P.x_gf : P.x_ga) + g * Hh + (fine ? i - Hh : i);
  {
    const uint4* src = a.uw + (size_t)k * (P.u_lds_w / 16);
    for (int q = tid; q < P.u_lds_w / 16; q += WR_THREADS) ((uint4*)lds)[q] = src[q];
    for (int c = tid; c < H; c += WR_THREADS) hv[c] = a.h_in ? xround(a.h_in[c]) : 0.0f;
    if (tid == 0) misc[0] = 0;
  }
  __syncthreads();
  float acc = 0.0f;
  const bool b44 = P.BW == 4;
  auto mac = [&](int r0, int n) {
    const int L = tid & 255;
    if (b44) {
      const uint2* wp = (const uint2*)wts + (size_t)r0 * 256 + L;
#pragma unroll 2
      for (int r = 0; r < n; ++r) {
        const int col0 = bix[((r0 + r) * BR + bro) * SL + part];
        const uint2 q = wp[r * 256];
        const float4 h4 = *(const float4*)(hv + col0);
        acc = __builtin_fmaf(bf_lo(q.x), h4.x, acc);
        acc = __builtin_fmaf(bf_hi(q.x), h4.y, acc);
        acc = __builtin_fmaf(bf_lo(q.y), h4.z, acc);
        acc = __builtin_fmaf(bf_hi(q.y), h4.w, acc);
      }
    } else {   // quads of slots: 4 weights, 4 indices per read (n, r0 multiples of 4)
      const uint2* wq = (const uint2*)wts + (size_t)(r0 / 4) * 256 + L;
      const uint2* iq = (const uint2*)bix + ((size_t)(r0 / 4) * BR + bro) * SL + part;
#pragma unroll 2
      for (int q = 0; q < n / 4; ++q) {
        const uint2 w4 = wq[q * 256];
        const uint2 i4 = iq[q * BR * SL];
        acc = __builtin_fmaf(bf_lo(w4.x), hv[i4.x & 0xffffu], acc);
        acc = __builtin_fmaf(bf_hi(w4.x), hv[i4.x >> 16], acc);
        acc = __builtin_fmaf(bf_lo(w4.y), hv[i4.y & 0xffffu], acc);
        acc = __builtin_fmaf(bf_hi(w4.y), hv[i4.y >> 16], acc);
      }
    }
  };
  // coarse columns [0, Hh)
  auto phase_c = [&]() {
    acc = 0.0f;
    if (cw) mac(0, NRC);
  };
  // fine columns [Hh, H); then the SL lanes of a row add up and the first publishes
  auto phase_f = [&](uint32_t tag, float cbv) {
    if (!cw) return;
    mac(NRC, NRF);
    float v = acc;
    for (int m = 1; m < SL; m <<= 1) v += __shfl_xor(v, m);
    if (lead) xpub(dst, tag, g < 2 ? v + cbv : v);   // bias + conditioning of the u and r gates
  };
  __builtin_amdgcn_s_waitcnt(0);   // records and h are in before the loop (see head_role)
  phase_c();
  phase_f(1u, lead && g < 2 ? cb_row(a, a.t0)[row] : 0.0f);
  const xw* YC = a.xc + P.x_yc;
  const xw* YF = a.xc + P.x_yf;
  // Wait for a half of h: lane jj of wave 4 watches the last word of head
  // jj's slice, then waves 4-7 read every word once into hv.
  auto gather_half = [&](const xw* Y, uint32_t tag, float* out, bool flags) {
    if (flags) {
      if (wave == 4) {
        float y;
        const int hj = lane < P.NK ? lane : 0;
        if (!poll_sleepy(Y + P.HR * hj + P.HR - 1, tag, &y, a)) misc[0] = 1;
      }
      __syncthreads();
      if (misc[0]) return;
    }
    if (!cw) {
      constexpr int MW = 8;                       // Hh <= 2048
      const int r = tid - 256;
      uint32_t pending = 0;
      float y[MW];
#pragma unroll
      for (int m = 0; m < MW; ++m) {
        y[m] = 0.0f;
        if (r + 256 * m < Hh) pending |= 1u << m;
      }
      WaitBudget wb{wr_clock(), 0};
      while (pending) {
        xw w[MW];
#pragma unroll
        for (int m = 0; m < MW; ++m) w[m] = (pending >> m & 1u) ? xpeek(Y + r + 256 * m) : 0;
#pragma unroll
        for (int m = 0; m < MW; ++m)
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
      for (int m = 0; m < MW; ++m)
        if (r + 256 * m < Hh) out[r + 256 * m] = y[m];
    }
    __syncthreads();
  };
  for (int64_t t = 0; t + 1 < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    const float cbv = lead && g < 2 ? cb_row(a, a.t0 + t + 1)[row] : 0.0f;
    gather_half(YC, tag, hv, true);
    if (misc[0]) return;
    phase_c();
    gather_half(YF, tag, hv + Hh, false);
    if (misc[0]) return;
    if (k == 0 && tid == 0) trace_at(a, t + 1, 11);
    phase_f(tag + 1, cbv);
    if (k == 0 && tid == 0) trace_at(a, t + 1, 12);
  }
}

template <int KH, int GU>
__global__ __launch_bounds__(WR_THREADS, 1) void wr_sparse_kernel(PersistArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int r = wr_role(a.P, blockIdx.x);
  if (r < 0) return;
  if (r < a.P.NH) head_role<KH, 4, GU, true>(a, r, lds);
  else sparse_unit_role(a, r - a.P.NH, lds);
}

// Bias + conditioning of every gate row for every frame of every stream
// (Sec. 2 conditioning): cb[s][f][row] = sum_q W_cond[row][q] feat[s][f][q]
// (fma chain in q order) + b[row].
extern "C" __global__ void wr_cond_kernel(const float* Wc, const float* bias, const float* feat, int Dc, int rows,
                                          int64_t n_frames, int n_streams, float* cb) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n_streams * n_frames * rows) return;
  const int64_t sf = idx / rows;                  // stream * n_frames + frame
  const int row = (int)(idx % rows);
  float acc = 0.0f;
  if (Dc > 0) {
    const float* w = Wc + (size_t)row * Dc;
    const float* x = feat + (size_t)sf * Dc;
    for (int q = 0; q < Dc; ++q) acc = __builtin_fmaf(w[q], x[q], acc);
    acc = acc + bias[row];
  } else {
    acc = bias[row];
  }
  cb[idx] = acc;
}

extern "C" __global__ void wr_fill_u64(u64* p, int64_t n, u64 v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

const void* wr_persist_kernel_ptr(int KH) {
  switch (KH) {
    case 1: return (const void*)wr_persist_kernel<1>;
    case 2: return (const void*)wr_persist_kernel<2>;
    case 3: return (const void*)wr_persist_kernel<3>;
    case 4: return (const void*)wr_persist_kernel<4>;
    case 7: return (const void*)wr_persist_kernel<7>;
    default: return nullptr;
  }
}
const void* wr_sparse_kernel_ptr(int KH, int GU) {
  switch (KH * 4 + GU) {
    case 1 * 4 + 1: return (const void*)wr_sparse_kernel<1, 1>;
    case 2 * 4 + 1: return (const void*)wr_sparse_kernel<2, 1>;
    case 4 * 4 + 1: return (const void*)wr_sparse_kernel<4, 1>;
    case 7 * 4 + 1: return (const void*)wr_sparse_kernel<7, 1>;
    case 8 * 4 + 2: return (const void*)wr_sparse_kernel<8, 2>;
    case 16 * 4 + 3: return (const void*)wr_sparse_kernel<16, 3>;
    default: return nullptr;
  }
}
const void* wr_cond_kernel_ptr() { return (const void*)wr_cond_kernel; }
const void* wr_fill_kernel_ptr() { return (const void*)wr_fill_u64; }
