// Pieces of the persistent batch-1 kernel shared by its plain and fused
// (Fused Subscale WaveRNN 2x, Sec. 4.4) variants: the bias + conditioning
// rows and the unit workgroups (R h of the whole state).
#pragma once
#include "wr_kern.h"
#include "wr_layout.h"
#include "wr_args.h"

// Row of the bias + conditioning table used at absolute sample n.
__device__ __forceinline__ const float* cb_row(const PersistArgs& a, int64_t n) {
  int64_t fr = n / a.frame_len;
  if (fr >= a.n_cb) fr = a.n_cb - 1;
  return a.cb + (size_t)fr * 3 * a.P.H;
}

// Fused 2x schedule (Sec. 4.2 horizon F): position of sub-tensor s at step
// t, and the sample whose conditioning frame it uses there (its first or
// last while idle).
__device__ __forceinline__ int64_t fused_pos(const PersistArgs& a, int s, int64_t t) {
  return t - (int64_t)s * (a.F + 1);
}
__device__ __forceinline__ int64_t fused_sample(const PersistArgs& a, int s, int64_t t) {
  int64_t p = fused_pos(a, s, t);
  p = p < 0 ? 0 : p >= a.rows ? a.rows - 1 : p;
  return 2 * p + s;
}

// ------------------------------------------------------------------ unit role
// Wave q < UCT owns coarse row tile k*UCT + q and wave 4 + q fine row tile
// k*UCT + q: coarse columns from LDS (used when y_c arrives), fine columns from
// VGPRs (used when y_f arrives, so the part on the way to the heads reads no
// weights from LDS); each publishes its 16 pre-activations once y_f is in.
// MR (mirrors form the coarse rows' fine-column products): a coarse wave
// publishes its coarse columns' part (with bias + conditioning) as soon as
// y_c is in and holds no fine columns; the fine rows' words go to the buffer
// of their step's parity (wr_dbuf), since mirrors read them too.
template <int KH, bool FUSED, bool MR = false>
__device__ __forceinline__ void unit_role(const PersistArgs& a, int k, unsigned char* lds) {
  constexpr int KT = 2 * KH;
  const PersistPlan& P = a.P;
  const int H = P.H, Hh = P.Hh, UCT = P.UCT;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const unsigned char* WC = lds;                                 // [UCT][KT] coarse tiles, coarse columns
  const unsigned char* WF = lds + UCT * KT * WR_FRAG;            // [UCT][KT] fine tiles, coarse columns
  unsigned char* img = lds + P.u_lds_w;                          // [2KT] operand image of h
  int* misc = (int*)(img + 2 * KT * WR_FRAG);
  const bool cw = wave < UCT, fw = wave >= 4 && wave - 4 < UCT;
  const bool fx = MR ? fw : (cw || fw);                           // waves with fine-column products
  const int q = cw ? wave : wave - 4;
  // this wave's tile: gate g, units i0 .. i0+15 of its half
  const int tile = k * UCT + q;
  const int g = tile / (Hh / 16), i0 = 16 * (tile % (Hh / 16));
  const int row = g * H + (fw ? Hh : 0) + i0 + (lane & 15);     // R row of lane n < 16
  xw* dst = a.xc + (fw ? P.x_gf : P.x_ga) + g * Hh + i0 + lane;
  {
    const uint4* src = a.uw + (size_t)k * (P.u_lds_w / 16);
    for (int i = tid; i < P.u_lds_w / 16; i += WR_THREADS) ((uint4*)lds)[i] = src[i];
    for (int i = tid; i < 2 * KT * WR_FRAG / 16; i += WR_THREADS) ((uint4*)img)[i] = uint4{0, 0, 0, 0};
    if (tid == 0) misc[0] = 0;
  }
  bf16x8 WR[KT];
  if (fx) {
    const uint4* src = a.ur + ((size_t)(fw ? P.NU * UCT + tile : tile) * KT) * 64 + lane;
#pragma unroll
    for (int i = 0; i < KT; ++i) WR[i] = __builtin_bit_cast(bf16x8, src[(size_t)i * 64]);
  }
  __syncthreads();
  for (int i = tid; i < H; i += WR_THREADS) {
    const float y = a.h_in ? xround(a.h_in[i]) : 0.0f;   // as the heads' exchanged h
    aput(img + (i >> 5) * WR_FRAG, i & 31, y);
  }
  __syncthreads();
  f32x4 acc0, acc1;
  // columns [0, KT) of the image: coarse inputs
  auto phase_c = [&]() {
    acc0 = f32x4{0, 0, 0, 0};
    acc1 = f32x4{0, 0, 0, 0};
    const unsigned char* W = (cw ? WC : WF) + q * KT * WR_FRAG;
    if (cw || fw) {
#pragma unroll
      for (int i = 0; i < KT; i += 2) {
        acc0 = mfma(afrag(img, i), *(const bf16x8*)(W + i * WR_FRAG + lane * 16), acc0);
        if (i + 1 < KT) acc1 = mfma(afrag(img, i + 1), *(const bf16x8*)(W + (i + 1) * WR_FRAG + lane * 16), acc1);
      }
    }
  };
  // MR: a coarse wave's words of step s (its coarse columns' part) once y_c is in
  auto publish_c = [&](int64_t s, float cbv) {
    if (MR && cw && lane < 16) {
      float v = mfma_row(acc0) + mfma_row(acc1);
      if (g < 2) v += cbv;                      // bias + conditioning of the u and r gates
      xpub(dst, (uint32_t)s + 1u, v);
    }
  };
  // columns [KT, 2KT): fine inputs; then publish the words of step s
  auto phase_f = [&](int64_t s, float cbv) {
    if (fx) {
#pragma unroll
      for (int i = 0; i < KT; i += 2) {
        acc0 = mfma(afrag(img, KT + i), WR[i], acc0);
        if (i + 1 < KT) acc1 = mfma(afrag(img, KT + i + 1), WR[i + 1], acc1);
      }
    }
    if (fx && lane < 16) {
      float v = mfma_row(acc0) + mfma_row(acc1);
      if (g < 2) v += cbv;                      // bias + conditioning of the u and r gates
      if (MR) xpub(dst + wr_dbuf(s, P.x_gfs), wr_dtag(s, P.x_gfs), v);
      else xpub(dst, (uint32_t)s + 1u, v);
    }
  };
  __builtin_amdgcn_s_waitcnt(0);   // weights and operands are in before the loop (see head_role)
  // step 0's pre-activations from the initial state
  phase_c();
  // the sample whose frame this lane's row uses at step t: the fused model's
  // quarter of sub-tensor s follows the sample its sub-tensor makes
  const int rs = (i0 + (lane & 15)) / (Hh / 2);
  auto cbs = [&](int64_t t) { return FUSED ? fused_sample(a, rs, t) : a.t0 + t; };
  {
    const float cb0 = (cw || fw) && g < 2 ? cb_row(a, cbs(0))[row] : 0.0f;
    publish_c(0, cb0);
    phase_f(0, cb0);
  }
  const xw* YC = a.xc + P.x_yc;
  const xw* YF = a.xc + P.x_yf;
  // Wait for a half of h.  Waves 3 and 7 own no row tile and never store, so
  // their loads do not wait for the publishing waves' store acknowledgements:
  // lane jj of wave 3 watches the last word of head jj's slice (little polling
  // traffic while the heads exchange logits), then waves 3 and 7 read every
  // word once and write operand tiles kt0 ...
  const bool reader = wave == 3 || wave == 7;
  auto gather_half = [&](const xw* Y, uint32_t tag, int kt0, bool flags) {
    if (flags) {
      if (wave == 3) {
        float y;
        const int hj = lane < P.NH ? lane : 0;
        if (!poll_sleepy(Y + 64 * hj + 63, tag, &y, a)) misc[0] = 1;
      }
      __syncthreads();
      if (misc[0]) return;
    }
    if (reader) {   // words 4 q .. 4 q + 3 (one head's) per 16-byte load, q = lane of the two waves
      const int q = (wave == 3 ? 0 : 64) + lane;
      if (4 * q < Hh) {
        WaitBudget wb{wr_clock(), 0};
        xw4 w;
        for (;;) {
          w = xpeek4(xrsrc(xopaque(Y), (uint32_t)Hh * 4u), 16u * q);
          if (xok4(w, tag)) break;
          if (!wait_ok(wb, a.err, a.limit, a.err)) {
            misc[0] = 1;
            break;
          }
        }
        const int i = 4 * q;
        unsigned char* f = img + (kt0 + (i >> 5)) * WR_FRAG;
        aput(f, i & 31, xval(w.x));
        aput(f, (i & 31) + 1, xval(w.y));
        aput(f, (i & 31) + 2, xval(w.z));
        aput(f, (i & 31) + 3, xval(w.w));
      }
    }
    __syncthreads();
  };
  for (int64_t t = 0; t + 1 < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    // bias + conditioning of this lane's row for the next step, loaded early
    const float cbv = (cw || fw) && lane < 16 && g < 2 ? cb_row(a, cbs(t + 1))[row] : 0.0f;
    gather_half(YC, tag, 0, true);
    if (misc[0]) return;
    if (k == 0 && tid == 0) trace_at(a, t, 20);
    phase_c();
    publish_c(t + 1, cbv);
    if (k == 0 && tid == 0) trace_at(a, t, 21);
    gather_half(YF, tag, KT, false);   // y_f gates the next coarse step: no flag phase
    if (misc[0]) return;
    if (k == 0 && tid == 0) trace_at(a, t + 1, 11);
    phase_f(t + 1, cbv);
    if (k == 0 && tid == 0) trace_at(a, t + 1, 12);
  }
}

