// Fused Subscale WaveRNN 2x (Sec. 4.4) on the persistent multi-workgroup kernel.
//
// Two sub-tensors share one WaveRNN by splitting its state: units [0, Q) are
// the coarse quarter of sub-tensor 0, [Q, 2Q) the coarse quarter of
// sub-tensor 1, [2Q, 3Q) and [3Q, 4Q) their fine quarters (Q = H/4).  So the
// coarse half and the fine half are those of the batch-1 kernel, and the
// units (R h of the whole state) are the batch-1 units.  What changes is on
// the heads:
//   - inputs: the last sample (c, f) of both sub-tensors (I* columns 0-3)
//     reach every unit; the fine quarter of sub-tensor s also sees its own
//     coarse byte of this step (column 4 + s), the mask applied at pack time;
//   - output layers: one MLP per (level, sub-tensor), so O1 / O3 are block
//     diagonal over the two quarters of a half and O2 / O4 give 64 logits per
//     half: the high and low nibble (16 classes each) of both sub-tensors'
//     bytes;
//   - draws: the draw wave's four rows of 16 lanes draw the four nibbles of a
//     half at once, each row from its own Philox word;
//   - schedule: step t runs position t of sub-tensor 0 and position
//     t - (F + 1) of sub-tensor 1 (Sec. 4.2 horizon F); a sub-tensor outside
//     its positions draws nothing and keeps its last sample as input.
// Sample 2 i + s of the utterance is position i of sub-tensor s.
#include "wr_unit.h"

namespace {

// Four 16-way inverse-CDF draws, one per row of 16 lanes of a wave (lane l
// holds logit z of class l % 16 of row l / 16, the row's uniform u): the same
// rule as draw_wave on 16 classes.  Returns the row's class (or `forced` when
// >= 0) in every lane of the row; *lse = max z + log sum exp(z - max).
__device__ __forceinline__ int draw_rows16(float z, float u, int forced, float* lse) {
  const int l = threadIdx.x & 63, row0 = l & 48;
  float m = z;
#pragma unroll
  for (int k = 8; k >= 1; k >>= 1) m = fmaxf(m, __shfl_xor(m, k, 16));
  const float w = fexp(z - m);
  float incl = w;
  incl += dpp<0x111, 0xf, true>(0.0f, incl);   // row_shr:1
  incl += dpp<0x112, 0xf, true>(0.0f, incl);   // row_shr:2
  incl += dpp<0x114, 0xf, true>(0.0f, incl);   // row_shr:4
  incl += dpp<0x118, 0xf, true>(0.0f, incl);   // row_shr:8
  const float Z = __shfl(incl, row0 | 15, 64);
  *lse = m + __logf(Z);
  if (forced >= 0) return forced;
  const u64 rowm = 0xffffull << row0;
  int count = __popcll(__ballot(incl <= u * Z) & rowm);
  if (count == 16) {   // clamp to the row's last class with nonzero weight
    const u64 nz = __ballot(w > 0.0f) & rowm;
    count = nz ? 63 - __clzll(nz) - row0 : 15;
  }
  return count;
}

// Bias + conditioning row of sub-tensor s at step t: the frame of the sample
// it makes there (its first or last while idle).
__device__ __forceinline__ const float* fused_cb(const PersistArgs& a, int s, int64_t t) {
  return cb_row(a, fused_sample(a, s, t));
}

template <int KH>
__device__ __forceinline__ void fused_head_role(const PersistArgs& a, int j, unsigned char* lds) {
  constexpr int RT = 4, KC = 2, KT = KH * KC, HR = 16 * RT, KO = HR / 32, NK = 2 * KT / RT;
  constexpr int NH = NK, DW = 7, Hh = 32 * KT, Q = Hh / 2;
  const PersistPlan& P = a.P;
  const int H = P.H;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  unsigned char* imc = lds;                        // y_c operand image [KT]
  unsigned char* imf = imc + KT * WR_FRAG;         // y_f operand image [KT]
  unsigned char* imo = imf + KT * WR_FRAG;         // relu(first layer) image [KO]
  float* op = (float*)(imo + KO * WR_FRAG);        // [KC][HR] first-layer partials
  int* misc = (int*)(op + KC * HR);                // [0] abort [1], [2] c of this step (s = 0, 1)
                                                   // [4], [5] last c, [6], [7] last f
  float* uni = (float*)(misc + 16);                // [2][64][8] uniforms of a batch of 64 steps
  int* tgt = (int*)(uni + 2 * 64 * 8);             // [2][64][2] teacher-forcing targets

  for (int i = tid; i < (2 * KT + KO) * WR_FRAG / 16; i += WR_THREADS) ((uint4*)lds)[i] = uint4{0, 0, 0, 0};
  // fragments: W1 [KH] (O1 rows, block diagonal), W3 [KH] (O3), W2 [KO] (class
  // tile `wave` of O2 over this head's columns; waves 0-3), W4 [KO]
  bf16x8 W1[KH], W3[KH], W2[KO], W4[KO];
  {
    const uint4* src = a.hw + ((size_t)(j * 8 + wave) * P.hw_frags) * 64 + lane;
#pragma unroll
    for (int i = 0; i < KH; ++i) W1[i] = __builtin_bit_cast(bf16x8, src[(size_t)i * 64]);
#pragma unroll
    for (int i = 0; i < KH; ++i) W3[i] = __builtin_bit_cast(bf16x8, src[(size_t)(KH + i) * 64]);
#pragma unroll
    for (int i = 0; i < KO; ++i) W2[i] = __builtin_bit_cast(bf16x8, src[(size_t)(2 * KH + i) * 64]);
#pragma unroll
    for (int i = 0; i < KO; ++i) W4[i] = __builtin_bit_cast(bf16x8, src[(size_t)(2 * KH + KO + i) * 64]);
  }
  // gate thread u < Hh: coarse unit u and fine unit Hh + u, both of sub-tensor sq.
  // I* columns: last c0, f0, c1, f1, then (fine rows) the own coarse byte.
  const bool gate = tid < Hh;
  const int u = tid, sq = u / Q;
  float ic[3][4], ifn[3][5];
  float hc = 0.0f, hf = 0.0f;
  if (gate) {
#pragma unroll
    for (int g = 0; g < 3; ++g) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        ic[g][q] = a.Iw[6 * (g * H + u) + q];
        ifn[g][q] = a.Iw[6 * (g * H + Hh + u) + q];
      }
      ifn[g][4] = a.Iw[6 * (g * H + Hh + u) + 4 + sq];
    }
    if (a.h_in) {
      hc = a.h_in[u];
      hf = a.h_in[Hh + u];
    }
  }
  const float b1r = tid < HR ? a.b1[j * HR + tid] : 0.0f;
  const float b3r = tid < HR ? a.b3[j * HR + tid] : 0.0f;
  const float b2l = wave == DW ? a.b2[lane] : 0.0f;     // 64 nibble-logit biases of a half
  const float b4l = wave == DW ? a.b4[lane] : 0.0f;
  if (tid < 2) {
    misc[4 + tid] = a.c_in ? a.c_in[tid] : 128;
    misc[6 + tid] = a.f_in ? a.f_in[tid] : 0;
    misc[1 + tid] = misc[4 + tid];
  }
  if (tid == 0) misc[0] = 0;
  const xw* GA = a.xc + P.x_ga;
  const xw* GF = a.xc + P.x_gf;
  xw* YC = a.xc + P.x_yc;
  xw* YF = a.xc + P.x_yf;
  xw* PCo = a.xc + P.x_pc + (size_t)j * P.x_ps;
  xw* PFo = a.xc + P.x_pf + (size_t)j * P.x_ps;
  const xw* PC = a.xc + P.x_pc;
  const xw* PF = a.xc + P.x_pf;
  const int rt = wave % RT, kc = wave / RT;
  xw pc[3] = {0, 0, 0}, pf[3] = {0, 0, 0};
  float cbe_c = 0.0f, cbe_f = 0.0f;
  auto prefetch_coarse = [&](int64_t t) {
    if (gate) {
      pc[0] = xpeek(GA + u); pc[1] = xpeek(GA + Hh + u); pc[2] = xpeek(GA + 2 * Hh + u);
      cbe_c = fused_cb(a, sq, t)[2 * H + u];
    }
  };
  auto prefetch_fine = [&](int64_t t) {
    if (gate) {
      pf[0] = xpeek(GF + u); pf[1] = xpeek(GF + Hh + u); pf[2] = xpeek(GF + 2 * Hh + u);
      cbe_f = fused_cb(a, sq, t)[2 * H + Hh + u];
    }
  };
  auto first_layer = [&](const bf16x8* W, const unsigned char* img, float b) {
    f32x4 acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < KH; i += 2) {
      acc0 = mfma(afrag(img, kc * KH + i), W[i], acc0);
      if (i + 1 < KH) acc1 = mfma(afrag(img, kc * KH + i + 1), W[i + 1], acc1);
    }
    if (lane < 16) op[kc * HR + 16 * rt + lane] = mfma_row(acc0) + mfma_row(acc1);
    __syncthreads();
    if (tid < HR) aput(imo + (tid >> 5) * WR_FRAG, tid & 31, wr_relu((op[tid] + op[HR + tid]) + b));
    __syncthreads();
  };
  // second layer: class tile `wave` (< 4) over this head's HR columns -> 16 of the 64 partials
  bool lx = false;   // all heads on one XCD: partials published into its L2
  auto second_layer = [&](const bf16x8* W, xw* dst, uint32_t tag) {
    if (wave >= 4) return;
    f32x4 A = {0, 0, 0, 0};
#pragma unroll
    for (int kt = 0; kt < KO; ++kt) A = mfma(afrag(imo, kt), W[kt], A);
    if (lane < 16) xpub_l(dst + 16 * wave + lane, tag, mfma_row(A), lx);
  };
  // the draw wave: lane l sums partial l of every head (in head order, as
  // every head does) once all carry `tag`; the first probe waits a little
  auto gather = [&](const xw* src, uint32_t tag, float* s) -> bool {
    __builtin_amdgcn_s_sleep(6);   // (measured: 2 x 64 clocks 7% slower)
    return sum_parts<NH>(src, P.x_ps, 0, NH, lane, tag, s, a);
  };
  // Philox blocks of steps t .. t+63 (both sub-tensors: counter (position, 2 u + s),
  // words 0-3 = coarse high, coarse low, fine high, fine low nibble) and targets
  auto fill_batch = [&](int64_t t, int b) {
    const int64_t st = t + lane;
    if (st < a.T) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int64_t p = fused_pos(a, s, st);
        const bool act = p >= 0 && p < a.rows;
        uint64_t w[4];
        wr_philox((uint64_t)(act ? p : 0), 2 * a.stream_id + s, 0, 0, a.seed, 0, w);
#pragma unroll
        for (int k = 0; k < 4; ++k) uni[(b * 64 + lane) * 8 + 4 * s + k] = (float)(uint32_t)(w[k] >> 40) * (1.0f / 16777216.0f);
        tgt[(b * 64 + lane) * 2 + s] = a.target && act ? a.target[2 * p + s] : 0;
      }
    }
  };
  if (wave == DW) fill_batch(0, 0);
  __syncthreads();
  prefetch_coarse(0);
  prefetch_fine(0);
  // coarse terms known before the last fine bytes: gate words, c columns
  float cu = 0.0f, cr = 0.0f, ce = 0.0f, cie = 0.0f;
  auto coarse_pre = [&](uint32_t tag, float xc0, float xc1, int64_t t) {
    if (!gate) return;
    __builtin_amdgcn_s_sleep(8);
    prefetch_coarse(t);
    const xw* ps[3] = {GA + u, GA + Hh + u, GA + 2 * Hh + u};
    float v[3];
    if (!poll_pref<3>(ps, pc, tag, v, a)) {
      misc[0] = 1;
      return;
    }
    cu = v[0] + __builtin_fmaf(ic[0][2], xc1, ic[0][0] * xc0);
    cr = v[1] + __builtin_fmaf(ic[1][2], xc1, ic[1][0] * xc0);
    ce = v[2];
    cie = __builtin_fmaf(ic[2][2], xc1, ic[2][0] * xc0);
  };
  // fine terms known before this step's coarse bytes: gate words, the four last-sample columns
  float fu = 0.0f, fr = 0.0f, fe = 0.0f, fie = 0.0f;
  auto fine_pre = [&](uint32_t tag, float xc0, float xf0, float xc1, float xf1) {
    if (!gate) return;
    const xw* ps[3] = {GF + u, GF + Hh + u, GF + 2 * Hh + u};
    float v[3];
    if (!poll_pref<3>(ps, pf, tag, v, a)) {
      misc[0] = 1;
      return;
    }
    auto last4 = [&](int g) {
      return __builtin_fmaf(ifn[g][3], xf1, __builtin_fmaf(ifn[g][2], xc1, __builtin_fmaf(ifn[g][1], xf0, ifn[g][0] * xc0)));
    };
    fu = v[0] + last4(0);
    fr = v[1] + last4(1);
    fe = v[2];
    fie = last4(2);
  };
  if (WR_LOCAL_XCHG) lx = leads_share_xcd(a.xc + P.x_xcc, P.NH, j, misc + 8, a);
  coarse_pre(1u, fscale(misc[4]), fscale(misc[5]), 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (misc[0]) return;

  // draw-wave state: this lane's row r = lane / 16 draws nibble (r & 1) of sub-tensor r / 2
  const int dr = lane >> 4, ds = dr >> 1, dpart = dr & 1;
  float zc_keep = 0.0f, tc = 0.0f;                  // coarse logit of this lane, row's coarse NLL term
  const bool trw = j == 0 && tid == DW * 64;        // tracing thread (draw wave)
  for (int64_t t = 0; t < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    if (trw) trace_at(a, t, 0);
    const int bs = (int)((t >> 6) & 1) * 64 + (int)(t & 63);
    if (wave == DW && (t & 63) == 0) fill_batch(t + 64, (int)(((t >> 6) + 1) & 1));
    const int64_t p0 = fused_pos(a, 0, t), p1 = fused_pos(a, 1, t);
    const bool act0 = p0 < a.rows, act1 = p1 >= 0;   // p0 >= 0 and p1 < rows at every step
    // (1) coarse gates of every unit, finished with the last fine bytes
    if (gate) {
      const float xf0 = fscale(misc[6]), xf1 = fscale(misc[7]);
      const float uu = fsig(__builtin_fmaf(ic[0][3], xf1, __builtin_fmaf(ic[0][1], xf0, cu)));
      const float rr = fsig(__builtin_fmaf(ic[1][3], xf1, __builtin_fmaf(ic[1][1], xf0, cr)));
      const float e = ftanh(__builtin_fmaf(rr, ce, __builtin_fmaf(ic[2][3], xf1, __builtin_fmaf(ic[2][1], xf0, cie)) + cbe_c));
      hc = __builtin_fmaf(uu, hc, (1.0f - uu) * e);
      aput(imc + (u >> 5) * WR_FRAG, u & 31, hc);
      if (u - HR * j < (unsigned)HR) xpub(YC + u, tag, hc);
    }
    __syncthreads();
    if (trw) trace_at(a, t, 1);
    // (2) coarse MLP slices of both sub-tensors -> 64 partial logits
    first_layer(W1, imc, b1r);
    second_layer(W2, PCo, tag);
    if (trw) trace_at(a, t, 3);
    if (t > 0) prefetch_fine(t);
    // (3) the draw wave sums the partials and draws the four coarse nibbles;
    // meanwhile the fine terms that do not need them
    if (wave == DW) {
      float s;
      if (!gather(PC, tag, &s)) misc[0] = 1;
      const float z = s + b2l;
      int forced = -1;
      if (a.target) forced = dpart ? (tgt[bs * 2 + ds] >> 8) & 15 : tgt[bs * 2 + ds] >> 12;
      float lse;
      const int nib = draw_rows16(z, uni[bs * 8 + 4 * ds + dpart], forced, &lse);
      zc_keep = z;
      tc = lse - __shfl(z, (lane & 48) + nib, 64);
      const int byte0 = 16 * __shfl(nib, 0, 64) + __shfl(nib, 16, 64);
      const int byte1 = 16 * __shfl(nib, 32, 64) + __shfl(nib, 48, 64);
      if (trw) trace_at(a, t, 16);
      if (lane == 0) {
        misc[1] = act0 ? byte0 : misc[4];
        misc[2] = act1 ? byte1 : misc[5];
      }
    } else {
      fine_pre(tag, fscale(misc[4]), fscale(misc[6]), fscale(misc[5]), fscale(misc[7]));
    }
    __syncthreads();
    if (misc[0]) return;
    if (trw) trace_at(a, t, 5);
    // (4) fine gates, each fine quarter with its own sub-tensor's coarse byte
    const int c0 = misc[1], c1 = misc[2];
    if (gate) {
      const float xo = fscale(sq ? c1 : c0);
      const float uu = fsig(__builtin_fmaf(ifn[0][4], xo, fu)), rr = fsig(__builtin_fmaf(ifn[1][4], xo, fr));
      const float e = ftanh(__builtin_fmaf(rr, fe, __builtin_fmaf(ifn[2][4], xo, fie) + cbe_f));
      hf = __builtin_fmaf(uu, hf, (1.0f - uu) * e);
      aput(imf + (u >> 5) * WR_FRAG, u & 31, hf);
      if (u - HR * j < (unsigned)HR) xpub(YF + u, tag, hf);
    }
    __syncthreads();
    if (trw) trace_at(a, t, 6);
    // (5) fine MLP slices -> 64 partial logits
    first_layer(W3, imf, b3r);
    second_layer(W4, PFo, tag);
    if (trw) trace_at(a, t, 8);
    // (6) fine nibbles, outputs; meanwhile the next step's coarse terms
    if (wave == DW) {
      float s;
      if (!gather(PF, tag, &s)) misc[0] = 1;
      const float z = s + b4l;
      int forced = -1;
      if (a.target) forced = dpart ? tgt[bs * 2 + ds] & 15 : (tgt[bs * 2 + ds] >> 4) & 15;
      float lse;
      const int nib = draw_rows16(z, uni[bs * 8 + 4 * ds + 2 + dpart], forced, &lse);
      const float tf = lse - __shfl(z, (lane & 48) + nib, 64);
      const int f0 = 16 * __shfl(nib, 0, 64) + __shfl(nib, 16, 64);
      const int f1 = 16 * __shfl(nib, 32, 64) + __shfl(nib, 48, 64);
      if (trw) trace_at(a, t, 18);
      const float rowt = tc + tf;                     // this row's two nibble terms
      const float nll = rowt + __shfl(rowt, lane + 16, 64);   // rows 2s and 2s + 1 (lanes 32 s)
      const bool act = ds ? act1 : act0;
      const int64_t p = ds ? p1 : p0;
      if (j == 0 && act) {
        const size_t o = (size_t)(2 * p + ds);
        if (a.zc_out) a.zc_out[o * 32 + (lane & 31)] = zc_keep;
        if (a.zf_out) a.zf_out[o * 32 + (lane & 31)] = z;
        if ((lane & 31) == 0) {
          const int cb_ = ds ? c1 : c0, fb = ds ? f1 : f0;
          if (a.out) a.out[o] = (uint16_t)(256 * cb_ + fb);
          if (a.nll_out) a.nll_out[o] = nll;
        }
      }
      if (lane == 0) {
        misc[4] = c0;                                 // an idle sub-tensor's c is its last c already
        misc[5] = c1;
        if (act0) misc[6] = f0;
        if (act1) misc[7] = f1;
      }
    } else if (t + 1 < a.T) {
      coarse_pre(tag + 1, fscale(c0), fscale(c1), t + 1);
    }
    __syncthreads();
    if (misc[0]) return;
    if (trw) trace_at(a, t, 10);
  }
  if (j == 0) {
    if (a.h_out && gate) {
      a.h_out[u] = hc;
      a.h_out[Hh + u] = hf;
    }
    if (tid < 2) {
      if (a.c_out) a.c_out[tid] = (uint8_t)misc[4 + tid];
      if (a.f_out) a.f_out[tid] = (uint8_t)misc[6 + tid];
    }
  }
}

}  // namespace

template <int KH>
__global__ __launch_bounds__(WR_THREADS, 1) void wr_fused_kernel(PersistArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int r = wr_role(a.P, blockIdx.x);
  if (r < 0) return;
  if (r < a.P.NH) fused_head_role<KH>(a, r, lds);
  else unit_role<KH, true>(a, r - a.P.NH, lds);
}

const void* wr_fused_kernel_ptr(int KH) {
  switch (KH) {
    case 1: return (const void*)wr_fused_kernel<1>;
    case 2: return (const void*)wr_fused_kernel<2>;
    case 3: return (const void*)wr_fused_kernel<3>;
    case 4: return (const void*)wr_fused_kernel<4>;
    case 7: return (const void*)wr_fused_kernel<7>;
    default: return nullptr;
  }
}
