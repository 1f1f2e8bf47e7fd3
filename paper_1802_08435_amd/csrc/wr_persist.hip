// Persistent multi-workgroup WaveRNN sampler (batch 1 per launch).
//
// The whole utterance runs inside one cooperative launch (Sec. 2.1): weights
// are loaded once into LDS, then every step runs the GRU of Eq. 2, the coarse
// head, the coarse draw, the fine half, the fine head and the fine draw.
// Workgroups exchange vectors through tagged 64-bit words (value + step tag)
// instead of grid-wide barriers, so each dependency costs one one-way hop:
//
//   U  (unit workgroups): R rows of their units, gate math, both draws
//   HC (coarse-head):     O1 rows + matching O2 columns -> partial coarse logits
//   HF (fine-head):       O3 rows + matching O4 columns -> partial fine logits
//
//   per step:  U --y_c--> HC --partials--> U (sum, draw c_t, fine gates)
//              U --y_f--> HF --partials--> U (sum, draw f_t, next coarse gates)
//
// R h_t is split by input half: R[:, coarse] y_c runs while the coarse head
// works, R[coarse rows, fine] y_f while the fine head works, and
// R[fine rows, fine] y_f after the next coarse gates (fine rows are needed
// only after c_{t+1} is drawn), so the matvec with R stays off the critical path.
#include "wr_device.h"
#include "wr_layout.h"
#include "wr_args.h"

// Partial matvec of one row-block over one input half.  Lane l = 8r + q:
// row r of the block, columns q*SEG .. q*SEG+SEG-1 of x.  Returns the full dot
// product of row r in all 8 lanes of its group.
template <int CPL>
__device__ __forceinline__ float rb_matvec(const uint4* W, const float* x) {
  const int lane = threadIdx.x & 63, q = lane & 7;
  const float* xq = x + q * (CPL * 8);
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    uint4 w = W[i * 64 + lane];
    float4 xa = *(const float4*)(xq + 8 * i);
    float4 xb = *(const float4*)(xq + 8 * i + 4);
    acc = __builtin_fmaf(bf_lo(w.x), xa.x, acc);
    acc = __builtin_fmaf(bf_hi(w.x), xa.y, acc);
    acc = __builtin_fmaf(bf_lo(w.y), xa.z, acc);
    acc = __builtin_fmaf(bf_hi(w.y), xa.w, acc);
    acc = __builtin_fmaf(bf_lo(w.z), xb.x, acc);
    acc = __builtin_fmaf(bf_hi(w.z), xb.y, acc);
    acc = __builtin_fmaf(bf_lo(w.w), xb.z, acc);
    acc = __builtin_fmaf(bf_hi(w.w), xb.w, acc);
  }
  acc += __shfl_xor(acc, 1, 64);
  acc += __shfl_xor(acc, 2, 64);
  acc += __shfl_xor(acc, 4, 64);
  return acc;
}

// Gather n tagged words into dst (all threads).  False on timeout / abort.
__device__ bool gather_words(const u64* src, int n, uint32_t tag, float* dst, const PersistArgs& a) {
  WaitBudget wb{wr_clock(), 0};
  const int nt = blockDim.x;
  int i0 = threadIdx.x, i1 = threadIdx.x + nt;
  bool p0 = i0 < n, p1 = i1 < n;
  while (p0 || p1) {
    u64 w0 = p0 ? xpeek(src + i0) : 0, w1 = p1 ? xpeek(src + i1) : 0;
    if (p0 && xtag(w0) == tag) { dst[i0] = xval(w0); p0 = false; }
    if (p1 && xtag(w1) == tag) { dst[i1] = xval(w1); p1 = false; }
    if ((p0 || p1) && !wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
  return true;
}

#define WR_MAXNC 16

// Phase timestamp of a traced step (one thread calls it).
__device__ __forceinline__ void trace_at(const PersistArgs& a, int64_t t, int slot) {
  if (a.trace && t < a.trace_steps) a.trace[t * WR_TRACE_SLOTS + slot] = wr_clock();
}

// Sum of the nparts partial logits of class v (fixed order) once all carry tag.
__device__ bool sum_partials(const u64* src, int nparts, int v, uint32_t tag, float* out, const PersistArgs& a) {
  WaitBudget wb{wr_clock(), 0};
  float vals[WR_MAXNC];
  uint32_t pending = (1u << nparts) - 1u;
  while (pending) {
    u64 w[WR_MAXNC];
#pragma unroll
    for (int j = 0; j < WR_MAXNC; ++j) w[j] = (pending >> j & 1u) ? xpeek(src + j * WR_CLASSES + v) : 0;
#pragma unroll
    for (int j = 0; j < WR_MAXNC; ++j)
      if ((pending >> j & 1u) && xtag(w[j]) == tag) {
        vals[j] = xval(w[j]);
        pending &= ~(1u << j);
      }
    if (pending && !wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
  float acc = 0.0f;
#pragma unroll
  for (int j = 0; j < WR_MAXNC; ++j)
    if (j < nparts) acc += vals[j];
  *out = acc;
  return true;
}

// Inverse-CDF draw over softmax(z) by one wave (4 classes per lane).
// Returns the class (or `forced` when >= 0); *lse = max z + log sum exp(z - max).
__device__ int draw_wave(const float* z, float u, int forced, float* lse) {
  const int l = threadIdx.x & 63;
  float4 z4 = *(const float4*)(z + 4 * l);
  float m = fmaxf(fmaxf(z4.x, z4.y), fmaxf(z4.z, z4.w));
  m = wave_max(m);
  float w0 = wr_exp(z4.x - m), w1 = wr_exp(z4.y - m), w2 = wr_exp(z4.z - m), w3 = wr_exp(z4.w - m);
  float s0 = w0, s1 = s0 + w1, s2 = s1 + w2, s3 = s2 + w3;
  float incl = s3;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    float o = __shfl_up(incl, d, 64);
    if (l >= d) incl += o;
  }
  float excl = __shfl_up(incl, 1, 64);
  if (l == 0) excl = 0.0f;
  float Z = __shfl(incl, 63, 64);
  *lse = m + logf(Z);
  if (forced >= 0) return forced;
  float thr = u * Z;
  int cnt = (excl + s0 <= thr) + (excl + s1 <= thr) + (excl + s2 <= thr) + (excl + s3 <= thr);
  int count = wave_sum_i(cnt);
  if (count == WR_CLASSES) {
    int last = w3 > 0.0f ? 4 * l + 3 : w2 > 0.0f ? 4 * l + 2 : w1 > 0.0f ? 4 * l + 1 : w0 > 0.0f ? 4 * l : -1;
    count = wave_max_i(last);
  }
  return count;
}

// ------------------------------------------------------------------ U role
template <int CPL>
__device__ void u_role(const PersistArgs& a, int k, unsigned char* lds) {
  const PersistPlan& P = a.P;
  const int H = P.H, Hh = P.Hh, UC = WR_UC;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const uint4* W = (const uint4*)lds;
  float* h = (float*)(lds + P.u_bytes);   // [H] current hidden state (gathered)
  float* Gc = h + H;                      // [3][UC] coarse rows: R h for the next coarse gates
  float* Gf = Gc + 3 * UC;                // [2][3][UC] fine rows, double-buffered by step parity
  float* add = Gf + 6 * UC;               // [6UC] by local row: bias + conditioning
  float* Iw = add + 6 * UC;               // [6UC][3]
  float* z = Iw + 18 * UC;                // [256]
  int* misc = (int*)(z + 256);            // [0] abort, [1] c_t, [2] f_t, [3] cprev, [4] fprev
  float* fmisc = (float*)(misc + 8);      // [0] uc, [1] uf, [2] lse_c, [3] z_c[c]
  // wave w < 3: coarse rows of gate w; w >= 3: fine rows of gate w - 3.
  const int g_w = wave % 3, half_w = wave / 3, rb_w = 2 * g_w + half_w;
  const int r_l = lane >> 3;
  auto grow = [&](int g, int half, int j) { return g * H + half * Hh + k * UC + j; };
  auto lrow = [&](int g, int half, int j) { return g * 2 * UC + half * UC + j; };

  {  // prologue: weights, I*, bias, state
    const uint4* src = a.wu + (size_t)k * (P.u_bytes / 16);
    uint4* dst = (uint4*)lds;
    for (int i = tid; i < P.u_bytes / 16; i += blockDim.x) dst[i] = src[i];
    for (int i = tid; i < H; i += blockDim.x) h[i] = a.h_in ? a.h_in[i] : 0.0f;
    for (int lr = tid; lr < 6 * UC; lr += blockDim.x) {
      int g = lr / (2 * UC), half = (lr / UC) & 1, j = lr % UC;
      int row = grow(g, half, j);
      Iw[3 * lr + 0] = a.Iw[3 * row + 0];
      Iw[3 * lr + 1] = a.Iw[3 * row + 1];
      Iw[3 * lr + 2] = a.Iw[3 * row + 2];
    }
    if (tid == 0) {
      misc[0] = 0;
      misc[3] = a.c_in ? a.c_in[0] : 128;
      misc[4] = a.f_in ? a.f_in[0] : 0;
    }
  }
  __syncthreads();
  {  // R h_0 for step 0: both halves
    float acc = rb_matvec<CPL>(W + (size_t)(0 * 6 + rb_w) * CPL * 64, h) +
                rb_matvec<CPL>(W + (size_t)(1 * 6 + rb_w) * CPL * 64, h + Hh);
    if ((lane & 7) == 0) {
      if (half_w == 0) Gc[g_w * UC + r_l] = acc;
      else Gf[0 * 3 * UC + g_w * UC + r_l] = acc;
    }
  }
  __syncthreads();

  u64* YC = a.xc + P.x_yc;
  u64* YF = a.xc + P.x_yf;
  const u64* PC = a.xc + P.x_pc;
  const u64* PF = a.xc + P.x_pf;
  int64_t cur_frame = -1;
  for (int64_t t = 0; t < a.T; ++t) {
    const int64_t n = a.t0 + t;
    const uint32_t tag = (uint32_t)(t + 1);
    const int par = (int)(t & 1);
    // [A] bias + conditioning of the frame
    int64_t fr = a.Dc > 0 ? n / a.frame_len : 0;
    if (a.Dc > 0 && fr >= a.n_frames) fr = a.n_frames - 1;
    if (fr != cur_frame) {
      cur_frame = fr;
      for (int lr = tid; lr < 6 * UC; lr += blockDim.x) {
        int g = lr / (2 * UC), half = (lr / UC) & 1, j = lr % UC;
        int row = grow(g, half, j);
        float v = a.bias[row];
        if (a.Dc > 0) {
          const float* wc = a.Wc + (size_t)row * a.Dc;
          const float* fv = a.feat + (size_t)fr * a.Dc;
          float acc = 0.0f;
          for (int q = 0; q < a.Dc; ++q) acc = __builtin_fmaf(wc[q], fv[q], acc);
          v = acc + v;
        }
        add[lr] = v;
      }
      __syncthreads();
    }
    const bool tr = k == 0 && tid == 0;                          // all phases of U workgroup 0
    const bool trl = k == P.NU - 1 && k > 0 && tid == 0;        // y_c published / gathered of the last
    if (tr) trace_at(a, t, 0);
    const float x0 = wr_scale(misc[3]), x1 = wr_scale(misc[4]);
    // [B] coarse gates of this workgroup's units -> publish y_c
    if (tid < UC) {
      const int j = tid, i = k * UC + j;
      float ix[3];
#pragma unroll
      for (int g = 0; g < 3; ++g) {
        const float* I = Iw + 3 * lrow(g, 0, j);
        ix[g] = __builtin_fmaf(I[1], x1, __builtin_fmaf(I[0], x0, 0.0f));
      }
      float au = Gc[0 * UC + j] + (ix[0] + add[lrow(0, 0, j)]);
      float ar = Gc[1 * UC + j] + (ix[1] + add[lrow(1, 0, j)]);
      float u = wr_sigmoid(au), r = wr_sigmoid(ar);
      float e = wr_tanh(__builtin_fmaf(r, Gc[2 * UC + j], ix[2] + add[lrow(2, 0, j)]));
      xpub(YC + i, tag, __builtin_fmaf(u, h[i], (1.0f - u) * e));
      if (tr) trace_at(a, t, 1);
      if (trl) trace_at(a, t, 25);
    }
    if (tid == 64) {
      float uc, uf;
      wr_uniforms(a.seed, a.stream_id, (uint64_t)n, &uc, &uf);
      fmisc[0] = uc;
      fmisc[1] = uf;
    }
    // [7b of step t-1] fine rows += R[fine rows, fine cols] y_f(t-1)
    if (t > 0 && half_w == 1) {
      float acc = rb_matvec<CPL>(W + (size_t)(1 * 6 + rb_w) * CPL * 64, h + Hh);
      if ((lane & 7) == 0) Gf[par * 3 * UC + g_w * UC + r_l] += acc;
    }
    // [C] gather y_c(t)
    if (!gather_words(YC, Hh, tag, h, a)) misc[0] = 1;
    __syncthreads();
    if (misc[0]) return;
    if (tr) trace_at(a, t, 2);
    if (trl) trace_at(a, t, 26);
    // [D] R[:, coarse cols] y_c(t): coarse rows -> Gc (next step), fine rows -> Gf[next]
    {
      float acc = rb_matvec<CPL>(W + (size_t)(0 * 6 + rb_w) * CPL * 64, h);
      if ((lane & 7) == 0) {
        if (half_w == 0) Gc[g_w * UC + r_l] = acc;
        else Gf[(par ^ 1) * 3 * UC + g_w * UC + r_l] = acc;
      }
      if (tr) trace_at(a, t, 3);
    }
    // [E] coarse logits = sum of head partials + b2, draw c_t
    const int64_t o = t;
    if (tid < WR_CLASSES) {
      float s;
      if (!sum_partials(PC, P.NC, tid, tag, &s, a)) misc[0] = 1;
      else z[tid] = s + a.b2[tid];
    }
    __syncthreads();
    if (misc[0]) return;
    if (tr) trace_at(a, t, 4);
    if (k == 0 && a.zc_out && tid < WR_CLASSES) a.zc_out[o * WR_CLASSES + tid] = z[tid];
    if (wave == 0) {
      float lse;
      int forced = a.target ? (a.target[o] >> 8) : -1;
      int c = draw_wave(z, fmisc[0], forced, &lse);
      if (lane == 0) {
        misc[1] = c;
        fmisc[2] = lse;
        fmisc[3] = z[c];
      }
    }
    __syncthreads();
    if (tr) trace_at(a, t, 5);
    const int c = misc[1];
    // [F] fine gates (c_t reaches the fine half only) -> publish y_f
    if (tid < UC) {
      const int j = tid, i = Hh + k * UC + j;
      const float x2 = wr_scale(c);
      const float* G = Gf + par * 3 * UC;
      float ix[3];
#pragma unroll
      for (int g = 0; g < 3; ++g) {
        const float* I = Iw + 3 * lrow(g, 1, j);
        ix[g] = __builtin_fmaf(I[2], x2, __builtin_fmaf(I[1], x1, __builtin_fmaf(I[0], x0, 0.0f)));
      }
      float au = G[0 * UC + j] + (ix[0] + add[lrow(0, 1, j)]);
      float ar = G[1 * UC + j] + (ix[1] + add[lrow(1, 1, j)]);
      float u = wr_sigmoid(au), r = wr_sigmoid(ar);
      float e = wr_tanh(__builtin_fmaf(r, G[2 * UC + j], ix[2] + add[lrow(2, 1, j)]));
      xpub(YF + (i - Hh), tag, __builtin_fmaf(u, h[i], (1.0f - u) * e));
      if (tr) trace_at(a, t, 6);
    }
    // [G] gather y_f(t)
    if (!gather_words(YF, Hh, tag, h + Hh, a)) misc[0] = 1;
    __syncthreads();
    if (misc[0]) return;
    if (tr) trace_at(a, t, 7);
    // [H] coarse rows += R[coarse rows, fine cols] y_f(t)
    if (half_w == 0) {
      float acc = rb_matvec<CPL>(W + (size_t)(1 * 6 + rb_w) * CPL * 64, h + Hh);
      if ((lane & 7) == 0) Gc[g_w * UC + r_l] += acc;
      if (tr) trace_at(a, t, 8);
    }
    // [I] fine logits, draw f_t
    if (tid < WR_CLASSES) {
      float s;
      if (!sum_partials(PF, P.NF, tid, tag, &s, a)) misc[0] = 1;
      else z[tid] = s + a.b4[tid];
    }
    __syncthreads();
    if (misc[0]) return;
    if (tr) trace_at(a, t, 9);
    if (k == 0 && a.zf_out && tid < WR_CLASSES) a.zf_out[o * WR_CLASSES + tid] = z[tid];
    if (wave == 0) {
      float lse;
      int forced = a.target ? (a.target[o] & 255) : -1;
      int f = draw_wave(z, fmisc[1], forced, &lse);
      if (lane == 0) {
        if (k == 0) {
          if (a.out) a.out[o] = (uint16_t)(256 * c + f);
          if (a.nll_out) a.nll_out[o] = (fmisc[2] - fmisc[3]) + (lse - z[f]);
        }
        misc[3] = c;
        misc[4] = f;
      }
    }
    __syncthreads();
    if (tr) trace_at(a, t, 10);
  }
  if (a.h_out && tid < UC) {
    a.h_out[k * UC + tid] = h[k * UC + tid];
    a.h_out[Hh + k * UC + tid] = h[Hh + k * UC + tid];
  }
  if (k == 0 && tid == 0) {
    if (a.c_out) a.c_out[0] = (uint8_t)misc[3];
    if (a.f_out) a.f_out[0] = (uint8_t)misc[4];
  }
}

// ------------------------------------------------------------------ head role
// First layer rows [j*HCR, +HCR) (padded to HCP), second layer columns of the
// same range: partial logits p[v] = sum_k O2[v][k] relu(O1[k] y + b1[k]).
template <int CPL>
__device__ void head_role(const PersistArgs& a, int j, bool fine, unsigned char* lds) {
  const PersistPlan& P = a.P;
  const int Hh = P.Hh, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const uint4* W1 = (const uint4*)lds;
  const uint4* W2 = (const uint4*)(lds + P.h1_bytes);
  float* y = (float*)(lds + P.h_bytes);
  float* o = y + Hh;
  float* b1s = o + P.HCP;
  int* misc = (int*)(b1s + P.HCP);
  {
    const uint4* src = (fine ? a.whf : a.whc) + (size_t)j * (P.h_bytes / 16);
    uint4* dst = (uint4*)lds;
    for (int i = tid; i < P.h_bytes / 16; i += blockDim.x) dst[i] = src[i];
    const float* b = fine ? a.b3 : a.b1;
    for (int r = tid; r < P.HCP; r += blockDim.x) b1s[r] = r < P.HCR ? b[j * P.HCR + r] : 0.0f;
    if (tid == 0) misc[0] = 0;
  }
  __syncthreads();
  const u64* Y = a.xc + (fine ? P.x_yf : P.x_yc);
  u64* PO = a.xc + (fine ? P.x_pf : P.x_pc) + (size_t)j * WR_CLASSES;
  const int nrb = P.HCP / 8;
  for (int64_t t = 0; t < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1);
    if (!gather_words(Y, Hh, tag, y, a)) misc[0] = 1;
    __syncthreads();
    if (misc[0]) return;
    const bool tr = j == 0 && tid == 0;
    const int ts = fine ? 20 : 16;
    if (tr) trace_at(a, t, ts);
    if (wave < nrb) {
      float acc = rb_matvec<CPL>(W1 + (size_t)wave * CPL * 64, y);
      if ((lane & 7) == 0) {
        int r = wave * 8 + (lane >> 3);
        o[r] = wr_relu(acc + b1s[r]);
      }
    }
    __syncthreads();
    if (tr) trace_at(a, t, ts + 1);
    if (tid < WR_CLASSES) {
      float acc = 0.0f;
      for (int kb = 0; kb < nrb; ++kb) {
        uint4 w = W2[kb * WR_CLASSES + tid];
        const float* ok = o + 8 * kb;
        acc = __builtin_fmaf(bf_lo(w.x), ok[0], acc);
        acc = __builtin_fmaf(bf_hi(w.x), ok[1], acc);
        acc = __builtin_fmaf(bf_lo(w.y), ok[2], acc);
        acc = __builtin_fmaf(bf_hi(w.y), ok[3], acc);
        acc = __builtin_fmaf(bf_lo(w.z), ok[4], acc);
        acc = __builtin_fmaf(bf_hi(w.z), ok[5], acc);
        acc = __builtin_fmaf(bf_lo(w.w), ok[6], acc);
        acc = __builtin_fmaf(bf_hi(w.w), ok[7], acc);
      }
      xpub(PO + tid, tag, acc);
      if (tr) trace_at(a, t, ts + 2);
    }
  }
}

template <int CPL>
__global__ __launch_bounds__(WR_THREADS, 1) void wr_persist_kernel(PersistArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int b = blockIdx.x, NU = a.P.NU, NC = a.P.NC;
  if (b < NU) u_role<CPL>(a, b, lds);
  else if (b < NU + NC) head_role<CPL>(a, b - NU, false, lds);
  else head_role<CPL>(a, b - NU - NC, true, lds);
}

extern "C" __global__ void wr_fill_u64(u64* p, int64_t n, u64 v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

template __global__ void wr_persist_kernel<1>(PersistArgs);
template __global__ void wr_persist_kernel<2>(PersistArgs);
template __global__ void wr_persist_kernel<3>(PersistArgs);
template __global__ void wr_persist_kernel<4>(PersistArgs);
template __global__ void wr_persist_kernel<5>(PersistArgs);
template __global__ void wr_persist_kernel<6>(PersistArgs);
template __global__ void wr_persist_kernel<7>(PersistArgs);
template __global__ void wr_persist_kernel<8>(PersistArgs);

// Host-side accessor so the launcher (host C++) can take the kernel address.
const void* wr_persist_kernel_ptr(int cpl) {
  switch (cpl) {
    case 1: return (const void*)wr_persist_kernel<1>;
    case 2: return (const void*)wr_persist_kernel<2>;
    case 3: return (const void*)wr_persist_kernel<3>;
    case 4: return (const void*)wr_persist_kernel<4>;
    case 5: return (const void*)wr_persist_kernel<5>;
    case 6: return (const void*)wr_persist_kernel<6>;
    case 7: return (const void*)wr_persist_kernel<7>;
    case 8: return (const void*)wr_persist_kernel<8>;
  }
  return nullptr;
}

const void* wr_fill_kernel_ptr() { return (const void*)wr_fill_u64; }
