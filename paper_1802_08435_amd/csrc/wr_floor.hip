// Synchronization floor of the persistent kernels: the same grid, roles and
// exchanged words per step as the batch-1 kernel of a plan (dense or
// block-sparse), with no arithmetic.  Per step and half each head publishes
// its slice of y and 256 partial logits and waits for the partials of every
// slice (the two all-reduces on the critical path of a step); it also reads
// the gate words of the half(s) it serves, without waiting, as the sampling
// kernel reads them ahead.  Each unit workgroup reads both halves of h from
// the heads and publishes its gate words for the next step.  With mirrors
// (the dense plan) each mirror waits for the coarse partials, publishes its
// words of the coarse rows for the next step and waits for the fine partials;
// the heads wait for those words at the start of a step, and the fine words
// and fine partials sit in the sampling kernel's two buffers; the partials and
// the mirrors' words stay in the L2 of the leads' XCD when all leads share
// one, as in the sampling kernels.  The time per
// step of this kernel is what the exchange pattern alone costs (Sec. 2.1 of
// the paper counts such a synchronization cost per step).
#include "wr_kern.h"

namespace {

__device__ __forceinline__ void floor_head(const PersistArgs& a, int j, unsigned char* lds) {
  const PersistPlan& P = a.P;
  const int Hh = P.Hh, NK = P.NK, HR = P.HR;
  const bool split = P.NH == 2 * NK;
  const bool coarse = !split || j < NK, fine = !split || j >= NK;
  const int jk = split ? j % NK : j;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  int* misc = (int*)lds;
  float* zs = (float*)(misc + 16);               // [2][256] logit sums (written, never read)
  const xw* GA = a.xc + P.x_ga;
  const xw* GF = a.xc + P.x_gf;
  const xw* HF = a.xc + P.x_hf;
  float* gsink = zs + 512;                       // [WR_THREADS] (written, never read)
  auto gsink_add = [&](float v) { gsink[tid] = v; };
  xw* YC = a.xc + P.x_yc;
  xw* YF = a.xc + P.x_yf;
  xw* PC = a.xc + P.x_pc;
  xw* PF = a.xc + P.x_pf;
  if (tid == 0) misc[0] = 0;
  __syncthreads();
  const bool lx = WR_LOCAL_XCHG && P.x_xcc &&
                  leads_share_xcd(a.xc + P.x_xcc, P.NH + P.NM, j, misc + 4, a);
  // with mirrors: wait for their words of the coarse rows (3 per unit)
  auto mirror_words = [&](uint32_t tag) {
    if (P.NM == 0 || tid >= Hh) return;
    const xw* ps[3] = {HF + tid, HF + Hh + tid, HF + 2 * Hh + tid};
    const xw w0[3] = {xpeek(ps[0]), xpeek(ps[1]), xpeek(ps[2])};
    float v[3];
    if (!poll_pref<3>(ps, w0, tag, v, a)) misc[0] = 1;
    else gsink_add(v[0] + v[1] + v[2]);
  };
  // gate words of every unit of a half (3 per unit), read once without waiting
  auto gate_words = [&](const xw* G) {
    float acc = 0.0f;
    for (int u = tid; u < Hh; u += WR_THREADS)
      acc += xval(xpeek(G + u)) + xval(xpeek(G + Hh + u)) + xval(xpeek(G + 2 * Hh + u));
    gsink[tid] = acc;
  };
  // partials of all NK slices: every wave first waits for the last word of
  // every slice, then thread (v, half) reads its half of the slices.  With
  // nothing to compute between the exchanges this is the least polling
  // traffic per exchange (the sampling kernel, which computes in between,
  // polls its words directly where there are few per thread: here that
  // would keep 512 threads per head polling all the time and measure the
  // polling load instead)
  auto gather = [&](const xw* src, uint32_t tag) {
    {
      float y;
      const int jj = lane < NK ? lane : 0;
      if (!poll_sleepy<false>(src + (size_t)jj * P.x_ps + 255, tag, &y, a)) misc[0] = 1;
    }
    const int v = tid & 255, hh = tid >> 8, h0 = (NK + 1) / 2;
    float s;
    if (!sum_parts<16>(src, P.x_ps, hh ? h0 : 0, hh ? NK : h0, v, tag, &s, a)) misc[0] = 1;
    else zs[hh * 256 + v] = s;
  };
  for (int64_t t = 0; t < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    if (coarse) mirror_words(tag);
    if (coarse && wave == 7)
      for (int i = lane; i < HR; i += 64) xpub(YC + HR * jk + i, tag, 0.0f);
    if (coarse && lane < 32) xpub_l(PC + (size_t)jk * P.x_ps + 32 * wave + lane, tag, 0.0f, lx);
    if (coarse) gate_words(GA);   // (read while the partials are exchanged, as the sampling heads prefetch)
    gather(PC, tag);
    __syncthreads();
    if (misc[0]) return;
    if (fine && wave == 7)
      for (int i = lane; i < HR; i += 64) xpub(YF + HR * jk + i, tag, 0.0f);
    xw* PFt = PF + wr_dbuf(t, P.x_pfs);
    const uint32_t ftag = wr_dtag(t, P.x_pfs);
    if (fine && lane < 32) xpub_l(PFt + (size_t)jk * P.x_ps + 32 * wave + lane, ftag, 0.0f, lx);
    if (fine) gate_words(GF + wr_dbuf(t, P.x_gfs));
    gather(PFt, ftag);
    __syncthreads();
    if (misc[0]) return;
  }
}

// A mirror: the coarse partials of step t, then its words of the coarse rows
// for step t + 1, then the fine partials of step t (reading the fine rows'
// words of step t meanwhile, without waiting).
__device__ __forceinline__ void floor_mirror(const PersistArgs& a, int j, unsigned char* lds) {
  const PersistPlan& P = a.P;
  const int Hh = P.Hh, NK = P.NK;
  const int tid = threadIdx.x, lane = tid & 63;
  constexpr int MRW = 16 * WR_MTILES;
  int* misc = (int*)lds;
  float* zs = (float*)(misc + 16);               // [2][256] logit sums, then [WR_THREADS] (written, never read)
  const xw* GF = a.xc + P.x_gf;
  const xw* PC = a.xc + P.x_pc;
  const xw* PF = a.xc + P.x_pf;
  xw* HF = a.xc + P.x_hf + (size_t)MRW * j;
  if (tid == 0) misc[0] = 0;
  __syncthreads();
  auto gather = [&](const xw* src, uint32_t tag) {
    {
      float y;
      const int jj = lane < NK ? lane : 0;
      if (!poll_sleepy<false>(src + (size_t)jj * P.x_ps + 255, tag, &y, a)) misc[0] = 1;
    }
    const int v = tid & 255, hh = tid >> 8, h0 = (NK + 1) / 2;
    float s;
    if (!sum_parts<16>(src, P.x_ps, hh ? h0 : 0, hh ? NK : h0, v, tag, &s, a)) misc[0] = 1;
    else zs[hh * 256 + v] = s;
  };
  const bool lx = WR_LOCAL_XCHG && leads_share_xcd(a.xc + P.x_xcc, P.NH + P.NM, P.NH + j, misc + 4, a);
  if (tid < MRW) xpub_l(HF + tid, 1u, 0.0f, lx);
  for (int64_t t = 0; t < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    gather(PC, tag);
    __syncthreads();
    if (misc[0]) return;
    if (t + 1 < a.T && tid < MRW) xpub_l(HF + tid, tag + 1, 0.0f, lx);
    {   // the fine rows' words of step t (read without waiting, while the fine partials are exchanged)
      const xw* G = GF + wr_dbuf(t, P.x_gfs);
      float acc = 0.0f;
      for (int u = tid; u < Hh; u += WR_THREADS)
        acc += xval(xpeek(G + u)) + xval(xpeek(G + Hh + u)) + xval(xpeek(G + 2 * Hh + u));
      zs[512 + tid] = acc;
    }
    gather(PF + wr_dbuf(t, P.x_pfs), wr_dtag(t, P.x_pfs));
    __syncthreads();
    if (misc[0]) return;
  }
}

__device__ __forceinline__ void floor_unit(const PersistArgs& a, int k, unsigned char* lds) {
  const PersistPlan& P = a.P;
  const int Hh = P.Hh, NK = P.NK, HR = P.HR;
  const int wpu = 3 * Hh / P.NU;                 // gate words of each half this unit publishes
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  int* misc = (int*)lds;
  float* hv = (float*)(misc + 16);               // [Hh] (written, never read)
  xw* GA = a.xc + P.x_ga + (size_t)k * wpu;
  xw* GF = a.xc + P.x_gf + (size_t)k * wpu;
  const xw* YC = a.xc + P.x_yc;
  const xw* YF = a.xc + P.x_yf;
  if (tid == 0) misc[0] = 0;
  __syncthreads();
  // the gate words of step s (the fine rows' in their buffer)
  auto publish_c = [&](int64_t s) {
    if (tid < wpu) xpub(GA + tid, (uint32_t)s + 1u, 0.0f);
  };
  auto publish_f = [&](int64_t s) {
    if (tid < wpu) xpub(GF + wr_dbuf(s, P.x_gfs) + tid, wr_dtag(s, P.x_gfs), 0.0f);
  };
  auto gather_half = [&](const xw* Y, uint32_t tag, bool flags) {
    if (flags) {
      if (wave == 4) {
        float y;
        const int hj = lane < NK ? lane : 0;
        if (!poll_sleepy(Y + HR * hj + HR - 1, tag, &y, a)) misc[0] = 1;
      }
      __syncthreads();
      if (misc[0]) return;
    }
    if (tid >= 256) {                            // all of a lane's words in flight at once
      constexpr int MW = 8;                      // Hh <= 2048
      const int r = tid - 256;
      uint32_t pending = 0;
#pragma unroll
      for (int m = 0; m < MW; ++m)
        if (r + 256 * m < Hh) pending |= 1u << m;
      WaitBudget wb{wr_clock(), 0};
      while (pending) {
        xw x[MW];
#pragma unroll
        for (int m = 0; m < MW; ++m) x[m] = (pending >> m & 1u) ? xpeek(Y + r + 256 * m) : 0;
#pragma unroll
        for (int m = 0; m < MW; ++m)
          if ((pending >> m & 1u) && xok(x[m], tag)) {
            hv[r + 256 * m] = xval(x[m]);
            pending &= ~(1u << m);
          }
        if (pending && !wait_ok(wb, a.err, a.limit, a.err)) {
          misc[0] = 1;
          break;
        }
      }
    }
    __syncthreads();
  };
  publish_c(0);
  publish_f(0);
  for (int64_t t = 0; t + 1 < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    gather_half(YC, tag, true);
    if (misc[0]) return;
    if (P.NM) publish_c(t + 1);                  // with mirrors: the coarse columns' part once y_c is in
    gather_half(YF, tag, false);
    if (misc[0]) return;
    if (!P.NM) publish_c(t + 1);
    publish_f(t + 1);
  }
}

}  // namespace

__global__ __launch_bounds__(WR_THREADS, 1) void wr_floor_kernel(PersistArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int r = wr_role(a.P, blockIdx.x);
  if (r < 0) return;
  if (r < a.P.NH) floor_head(a, r, lds);
  else if (r < a.P.NH + a.P.NM) floor_mirror(a, r - a.P.NH, lds);
  else floor_unit(a, r - a.P.NH - a.P.NM, lds);
}

const void* wr_floor_kernel_ptr() { return (const void*)wr_floor_kernel; }
