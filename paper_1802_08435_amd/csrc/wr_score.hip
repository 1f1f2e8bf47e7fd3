// Teacher-forced scoring of the dense batch-1 model (the NLL of Sec. 5 on
// given audio).  With every byte of every step given, a step only updates h
// (the gates of Eq. 2): no draw and no output layer sits in the serial loop,
// so one kind of workgroup does it all, with one exchange per step.
//
// Workgroup k owns hidden units 16 k .. 16 k + 15 (all in one half).  Waves
// 0-2 hold the tiles of its three gate rows of R (u, r, e) in VGPRs and form
// R h for them on the matrix cores; 16 lanes finish the gates with the given
// bytes and publish the new slice of h; waves 3-7 gather the next h from every
// workgroup into the operand image (an all-gather: one hop per step).  The
// products and the gate arithmetic are the sampling kernel's operation for
// operation, so a scored trajectory reproduces the sampler's state bit for
// bit: a fine row's R h is one pass over all columns (even and odd column
// tiles in two accumulation chains), a coarse row's is the sampling units'
// coarse-column part (two chains, + bias and conditioning) plus the sampling
// mirrors' fine-column part (one chain per half of the fine columns, the
// halves added), each rounded as the exchange delivers it (lowest bit
// cleared).  The output layers run
// afterwards over all steps at once (wr_cnn_gemm), and the NLL per step in
// wr_score_nll.
//
// Exchange: h_s goes to buffer s mod 2 of [2][H] words, tagged with the
// parity of its generation s / 2 + 1.  A workgroup writes h_{s+2} into a
// buffer only after it has read every workgroup's h_{s+1}, which each
// publishes only after reading all of h_s: no reader is overtaken, and the
// generation bit tells h_s from h_{s-2} in the same buffer.
#include "wr_kern.h"

namespace {

__device__ __forceinline__ const float* score_cb(const ScoreArgs& a, int64_t n) {
  int64_t fr = n / a.frame_len;
  if (fr >= a.n_cb) fr = a.n_cb - 1;
  return a.cb + (size_t)fr * 3 * a.H;
}

// The products of a gate wave's 16 rows with h (operand image img, fragments
// W over all KT2 column tiles).  Fine rows: even and odd column tiles in
// acc0 and acc1 (the sampling units' fine rows).  Coarse rows: the coarse
// column tiles in acc0 and acc1 (the units' coarse-column part), and the two
// halves of the fine column tiles in one chain each, accA and accB (the
// mirrors' waves, in column order).
template <int KT2>
__device__ __forceinline__ void score_products(const unsigned char* img, const bf16x8* W, bool fine, f32x4& acc0,
                                               f32x4& acc1, f32x4& accA, f32x4& accB) {
  constexpr int KT = KT2 / 2, MK = KT / 2;
  if (fine) {
#pragma unroll
    for (int i = 0; i < KT2; i += 2) {
      acc0 = mfma(afrag(img, i), W[i], acc0);
      if (i + 1 < KT2) acc1 = mfma(afrag(img, i + 1), W[i + 1], acc1);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < KT; i += 2) {
    acc0 = mfma(afrag(img, i), W[i], acc0);
    if (i + 1 < KT) acc1 = mfma(afrag(img, i + 1), W[i + 1], acc1);
  }
#pragma unroll
  for (int i = 0; i < MK; ++i) {
    accA = mfma(afrag(img, KT + i), W[KT + i], accA);
    accB = mfma(afrag(img, KT + MK + i), W[KT + MK + i], accB);
  }
}

}  // namespace

template <int KT2>
__global__ __launch_bounds__(WR_THREADS, 1) void wr_score_kernel(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  unsigned char* img = lds;                          // [KT2] operand image of h
  float* pre = (float*)(lds + KT2 * WR_FRAG);        // [3][16] this step's R h (+ bias, conditioning) of u, r, e
  int* misc = (int*)(pre + 48);                      // [0] abort
  constexpr int NG = WR_THREADS - 192;               // gathering lanes (waves 3-7)
  constexpr int MW4 = (8 * KT2 + NG - 1) / NG;       // 16-byte groups of h per gathering lane
  const int k = blockIdx.x, H = a.H, Hh = a.Hh;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  for (int i = tid; i < KT2 * WR_FRAG / 16; i += WR_THREADS) ((uint4*)img)[i] = uint4{0, 0, 0, 0};
  if (tid == 0) misc[0] = 0;
  bf16x8 W[KT2];
  if (wave < 3) {
    const uint4* src = a.w + ((size_t)(k * 3 + wave) * KT2) * 64 + lane;
#pragma unroll
    for (int i = 0; i < KT2; ++i) W[i] = __builtin_bit_cast(bf16x8, src[(size_t)i * 64]);
  }
  __syncthreads();
  for (int i = tid; i < H; i += WR_THREADS) aput(img + (i >> 5) * WR_FRAG, i & 31, a.h_in ? xround(a.h_in[i]) : 0.0f);
  // gate thread tid < 16: unit u, its I* row, its full-precision state and the last bytes
  const bool gt = tid < 16;
  const int u = 16 * k + (tid & 15);
  const bool fine = u >= Hh;
  float cf[3][3];
#pragma unroll
  for (int g = 0; g < 3; ++g)
#pragma unroll
    for (int q = 0; q < 3; ++q) cf[g][q] = gt ? a.Iw[3 * (g * H + u) + q] : 0.0f;
  float h = gt && a.h_in ? a.h_in[u] : 0.0f;
  int cp = a.c_in ? a.c_in[0] : 128, fp = a.f_in ? a.f_in[0] : 0;
  __builtin_amdgcn_s_waitcnt(0);   // prologue loads in before the loop (see the persistent heads)
  __syncthreads();
  for (int64_t s = 0; s < a.T; ++s) {
    if (s > 0) {   // h_{s-1} of every workgroup into the image
      if (wave >= 3) {   // 4 words (units 4 q .. 4 q + 3) per 16-byte load, each word checked
        const xw* Y = a.xc + (size_t)((s - 1) & 1) * H;
        const uint32_t tag = (uint32_t)((s - 1) >> 1) + 1u;
        const int r = tid - 192;
        uint32_t pending = 0;
#pragma unroll
        for (int m = 0; m < MW4; ++m)
          if (r + NG * m < H / 4) pending |= 1u << m;
        WaitBudget wb{wr_clock(), 0};
        while (pending) {
          const __amdgpu_buffer_rsrc_t rs = xrsrc(xopaque(Y), (uint32_t)H * 4u);
          xw4 w[MW4];
#pragma unroll
          for (int m = 0; m < MW4; ++m) w[m] = (pending >> m & 1u) ? xpeek4(rs, 16u * (r + NG * m)) : xw4{0, 0, 0, 0};
#pragma unroll
          for (int m = 0; m < MW4; ++m)
            if ((pending >> m & 1u) && xok4(w[m], tag)) {
              const int i = 4 * (r + NG * m);
              aput(img + (i >> 5) * WR_FRAG, i & 31, xval(w[m].x));
              aput(img + (i >> 5) * WR_FRAG, (i & 31) + 1, xval(w[m].y));
              aput(img + (i >> 5) * WR_FRAG, (i & 31) + 2, xval(w[m].z));
              aput(img + (i >> 5) * WR_FRAG, (i & 31) + 3, xval(w[m].w));
              pending &= ~(1u << m);
            }
          if (pending && !wait_ok(wb, a.err, a.limit, a.err)) {
            misc[0] = 1;
            break;
          }
        }
      }
      __syncthreads();
      if (misc[0]) return;
    }
    const int64_t n = a.t0 + s;
    if (wave < 3) {   // gate `wave`: rows wave H + 16 k .. + 15 of R h, as the sampling kernel forms them
      f32x4 acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0}, accA = {0, 0, 0, 0}, accB = {0, 0, 0, 0};
      score_products<KT2>(img, W, fine, acc0, acc1, accA, accB);
      if (lane < 16) {
        float v = mfma_row(acc0) + mfma_row(acc1);
        if (wave < 2) v += score_cb(a, n)[wave * H + 16 * k + lane];   // bias + conditioning of u and r
        pre[wave * 16 + lane] = fine ? xround(v) : xround(v) + xround(mfma_row(accA) + mfma_row(accB));
      }
    }
    __syncthreads();
    if (gt) {
      const float v0 = pre[tid], v1 = pre[16 + tid], v2 = pre[32 + tid];
      const float cbe = score_cb(a, n)[2 * H + u];
      const int tg = a.target[s], c = tg >> 8;
      const float x0 = fscale(cp), x1 = fscale(fp);
      if (!fine) {   // the sampling head's coarse terms, then its gates with f_{t-1}
        const float cu = v0 + cf[0][0] * x0, cr = v1 + cf[1][0] * x0, cie = cf[2][0] * x0;
        const float uu = fsig(__builtin_fmaf(cf[0][1], x1, cu)), rr = fsig(__builtin_fmaf(cf[1][1], x1, cr));
        const float e = ftanh(__builtin_fmaf(rr, v2, __builtin_fmaf(cf[2][1], x1, cie) + cbe));
        h = __builtin_fmaf(uu, h, (1.0f - uu) * e);
        a.traj_c[s * Hh + u] = h;
      } else {       // its fine terms, then its gates with c_t
        const float fu = v0 + __builtin_fmaf(cf[0][1], x1, cf[0][0] * x0);
        const float fr = v1 + __builtin_fmaf(cf[1][1], x1, cf[1][0] * x0);
        const float fie = __builtin_fmaf(cf[2][1], x1, cf[2][0] * x0);
        const float x2 = fscale(c);
        const float uu = fsig(__builtin_fmaf(cf[0][2], x2, fu)), rr = fsig(__builtin_fmaf(cf[1][2], x2, fr));
        const float e = ftanh(__builtin_fmaf(rr, v2, __builtin_fmaf(cf[2][2], x2, fie) + cbe));
        h = __builtin_fmaf(uu, h, (1.0f - uu) * e);
        a.traj_f[s * Hh + (u - Hh)] = h;
      }
      xpub(a.xc + (size_t)(s & 1) * H + u, (uint32_t)(s >> 1) + 1u, h);
      cp = c;
      fp = tg & 255;
    }
  }
  if (gt && a.h_out) a.h_out[u] = h;
  if (k == 0 && tid == 0) {
    if (a.c_out) a.c_out[0] = (uint8_t)cp;
    if (a.f_out) a.f_out[0] = (uint8_t)fp;
  }
}

// Up to 8 utterances at once (a.nv of them).  Vector b sits in rows 2b and
// 2b + 1 of the operand image, so the products cost what one utterance's do,
// and lane l of a gate wave's result holds output row l % 16 of vectors
// 2 (l / 16) and 2 (l / 16) + 1.  Thread 16 b + i (< 16 nv) finishes unit
// 16 k + i of vector b with wr_score_kernel's arithmetic (vector 0's
// products come from the same lanes and elements of the same products), so
// every utterance's state and logits are those of scoring it alone, bit for
// bit.  Exchange: h_s of vector b at xc[(s mod 2) 8H + b H + u], the tags as
// above; the gathering lanes read nv H words per step.
template <int KT2>
__global__ __launch_bounds__(WR_THREADS, 1) void wr_score_multi(ScoreArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  constexpr int H = 32 * KT2, LV = 8;
  unsigned char* img = lds;                          // [KT2] operand image of h (vector b: rows 2b, 2b + 1)
  float* pre = (float*)(lds + KT2 * WR_FRAG);        // [3][LV][16] this step's R h (+ bias, conditioning)
  int* misc = (int*)(pre + 3 * LV * 16);             // [0] abort
  constexpr int NG = WR_THREADS - 192;               // gathering lanes (waves 3-7)
  constexpr int MW4 = (LV * H / 4 + NG - 1) / NG;    // 16-byte groups per gathering lane at most
  static_assert(MW4 <= 32, "pending mask");
  const int k = blockIdx.x, Hh = a.Hh, nv = a.nv;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  for (int i = tid; i < KT2 * WR_FRAG / 16; i += WR_THREADS) ((uint4*)img)[i] = uint4{0, 0, 0, 0};
  if (tid == 0) misc[0] = 0;
  bf16x8 W[KT2];
  if (wave < 3) {
    const uint4* src = a.w + ((size_t)(k * 3 + wave) * KT2) * 64 + lane;
#pragma unroll
    for (int i = 0; i < KT2; ++i) W[i] = __builtin_bit_cast(bf16x8, src[(size_t)i * 64]);
  }
  __syncthreads();
  for (int i = tid; i < nv * H; i += WR_THREADS) {
    const int b = i / H, col = i % H;
    aput(img + (col >> 5) * WR_FRAG, col & 31, a.h_in ? xround(a.h_in[i]) : 0.0f, b);
  }
  // gate thread tid < 16 nv: unit u of vector ub, its I* row, its state and last bytes
  const int ub = tid >> 4;
  const bool gt = ub < nv;
  const int u = 16 * k + (tid & 15);
  const bool fine = u >= Hh;
  float cf[3][3];
#pragma unroll
  for (int g = 0; g < 3; ++g)
#pragma unroll
    for (int q = 0; q < 3; ++q) cf[g][q] = gt ? a.Iw[3 * (g * H + u) + q] : 0.0f;
  float h = gt && a.h_in ? a.h_in[(size_t)ub * H + u] : 0.0f;
  int cp = gt && a.c_in ? a.c_in[ub] : 128, fp = gt && a.f_in ? a.f_in[ub] : 0;
  const float* cbv = a.cb + (size_t)(gt ? ub : 0) * a.n_cb * 3 * H;   // this vector's table
  const uint16_t* tgv = a.target + (size_t)(gt ? ub : 0) * a.T;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int64_t s = 0; s < a.T; ++s) {
    if (s > 0) {   // h_{s-1} of every workgroup and vector into the image
      if (wave >= 3) {   // 4 words of one vector per 16-byte load, each word checked
        const xw* Y = a.xc + (size_t)((s - 1) & 1) * LV * H;
        const uint32_t tag = (uint32_t)((s - 1) >> 1) + 1u;
        const int r = tid - 192;
        uint32_t pending = 0;
#pragma unroll
        for (int m = 0; m < MW4; ++m)
          if (r + NG * m < nv * H / 4) pending |= 1u << m;
        WaitBudget wb{wr_clock(), 0};
        while (pending) {
          const __amdgpu_buffer_rsrc_t rs = xrsrc(xopaque(Y), (uint32_t)(LV * H) * 4u);
          xw4 w[MW4];
#pragma unroll
          for (int m = 0; m < MW4; ++m) w[m] = (pending >> m & 1u) ? xpeek4(rs, 16u * (r + NG * m)) : xw4{0, 0, 0, 0};
#pragma unroll
          for (int m = 0; m < MW4; ++m)
            if ((pending >> m & 1u) && xok4(w[m], tag)) {
              const int i = 4 * (r + NG * m), b = i / H, col = i % H;
              unsigned char* f = img + (col >> 5) * WR_FRAG;
              aput(f, col & 31, xval(w[m].x), b);
              aput(f, (col & 31) + 1, xval(w[m].y), b);
              aput(f, (col & 31) + 2, xval(w[m].z), b);
              aput(f, (col & 31) + 3, xval(w[m].w), b);
              pending &= ~(1u << m);
            }
          if (pending && !wait_ok(wb, a.err, a.limit, a.err)) {
            misc[0] = 1;
            break;
          }
        }
      }
      __syncthreads();
      if (misc[0]) return;
    }
    const int64_t n = a.t0 + s;
    int64_t fr = n / a.frame_len;
    if (fr >= a.n_cb) fr = a.n_cb - 1;
    if (wave < 3) {   // gate `wave`: rows wave H + 16 k .. + 15 of R h for every vector
      f32x4 acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0}, accA = {0, 0, 0, 0}, accB = {0, 0, 0, 0};
      score_products<KT2>(img, W, fine, acc0, acc1, accA, accB);
      const int b0 = 2 * (lane >> 4), row = lane & 15;
      if (b0 < nv) {
        float v0 = mfma_row(acc0) + mfma_row(acc1), v1 = mfma_row_hi(acc0) + mfma_row_hi(acc1);
        if (wave < 2) {   // bias + conditioning of u and r
          v0 += a.cb[((size_t)b0 * a.n_cb + fr) * 3 * H + wave * H + 16 * k + row];
          if (b0 + 1 < nv) v1 += a.cb[((size_t)(b0 + 1) * a.n_cb + fr) * 3 * H + wave * H + 16 * k + row];
        }
        const float f0 = fine ? 0.0f : xround(mfma_row(accA) + mfma_row(accB));
        const float f1 = fine ? 0.0f : xround(mfma_row_hi(accA) + mfma_row_hi(accB));
        pre[(wave * LV + b0) * 16 + row] = fine ? xround(v0) : xround(v0) + f0;
        if (b0 + 1 < nv) pre[(wave * LV + b0 + 1) * 16 + row] = fine ? xround(v1) : xround(v1) + f1;
      }
    }
    __syncthreads();
    if (gt) {
      const int ui = tid & 15;
      const float v0 = pre[ub * 16 + ui], v1 = pre[(LV + ub) * 16 + ui], v2 = pre[(2 * LV + ub) * 16 + ui];
      const float cbe = cbv[fr * 3 * H + 2 * H + u];
      const int tg = tgv[s], c = tg >> 8;
      const float x0 = fscale(cp), x1 = fscale(fp);
      if (!fine) {
        const float cu = v0 + cf[0][0] * x0, cr = v1 + cf[1][0] * x0, cie = cf[2][0] * x0;
        const float uu = fsig(__builtin_fmaf(cf[0][1], x1, cu)), rr = fsig(__builtin_fmaf(cf[1][1], x1, cr));
        const float e = ftanh(__builtin_fmaf(rr, v2, __builtin_fmaf(cf[2][1], x1, cie) + cbe));
        h = __builtin_fmaf(uu, h, (1.0f - uu) * e);
        a.traj_c[((size_t)ub * a.T + s) * Hh + u] = h;
      } else {
        const float fu = v0 + __builtin_fmaf(cf[0][1], x1, cf[0][0] * x0);
        const float fr2 = v1 + __builtin_fmaf(cf[1][1], x1, cf[1][0] * x0);
        const float fie = __builtin_fmaf(cf[2][1], x1, cf[2][0] * x0);
        const float x2 = fscale(c);
        const float uu = fsig(__builtin_fmaf(cf[0][2], x2, fu)), rr = fsig(__builtin_fmaf(cf[1][2], x2, fr2));
        const float e = ftanh(__builtin_fmaf(rr, v2, __builtin_fmaf(cf[2][2], x2, fie) + cbe));
        h = __builtin_fmaf(uu, h, (1.0f - uu) * e);
        a.traj_f[((size_t)ub * a.T + s) * Hh + (u - Hh)] = h;
      }
      xpub(a.xc + (size_t)(s & 1) * LV * H + (size_t)ub * H + u, (uint32_t)(s >> 1) + 1u, h);
      cp = c;
      fp = tg & 255;
    }
  }
  if (gt && a.h_out) a.h_out[(size_t)ub * H + u] = h;
  if (k == 0 && gt && (tid & 15) == 0) {
    if (a.c_out) a.c_out[ub] = (uint8_t)cp;
    if (a.f_out) a.f_out[ub] = (uint8_t)fp;
  }
}

// NLL of each scored step from its logits: (lse z_c - z_c[c]) + (lse z_f - z_f[f]),
// one wave per row, with the draw's reduction (max, hardware exp2, sum, log).
extern "C" __global__ void wr_score_nll(const float* zc, const float* zf, const uint16_t* target, int64_t rows,
                                        float* nll) {
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int l = threadIdx.x & 63, tg = target[row];
  float r[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const float* z = (q ? zf : zc) + row * 256;
    const float4 z4 = *(const float4*)(z + 4 * l);
    const float mx = wave_maxf(fmaxf(fmaxf(z4.x, z4.y), fmaxf(z4.z, z4.w)));
    float sm = fexp(z4.x - mx) + fexp(z4.y - mx) + fexp(z4.z - mx) + fexp(z4.w - mx);
    for (int o = 32; o >= 1; o >>= 1) sm += __shfl_xor(sm, o, 64);
    r[q] = (mx + __logf(sm)) - z[q ? (tg & 255) : (tg >> 8)];
  }
  if (l == 0) nll[row] = r[0] + r[1];
}

const void* wr_score_kernel_ptr(int KT2) {
  switch (KT2) {
    case 4: return (const void*)wr_score_kernel<4>;
    case 8: return (const void*)wr_score_kernel<8>;
    case 12: return (const void*)wr_score_kernel<12>;
    case 16: return (const void*)wr_score_kernel<16>;
    case 28: return (const void*)wr_score_kernel<28>;
    default: return nullptr;
  }
}
const void* wr_score_multi_ptr(int KT2) {
  switch (KT2) {
    case 4: return (const void*)wr_score_multi<4>;
    case 8: return (const void*)wr_score_multi<8>;
    case 12: return (const void*)wr_score_multi<12>;
    case 16: return (const void*)wr_score_multi<16>;
    case 28: return (const void*)wr_score_multi<28>;
    default: return nullptr;
  }
}
const void* wr_score_nll_ptr() { return (const void*)wr_score_nll; }
