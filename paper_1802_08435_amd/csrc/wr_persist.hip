// Persistent multi-workgroup WaveRNN sampler (batch 1 per launch).
//
// The whole utterance runs inside one cooperative launch (Sec. 2.1): weights
// are loaded once into LDS, and every step evaluates the GRU of Eq. 2, the
// coarse head, the coarse draw, the fine half, the fine head and the fine draw.
// Workgroups exchange vectors through tagged 64-bit words (value + step tag)
// instead of grid-wide barriers: each dependency costs one one-way hop.
//
// Critical path per step, all inside the NH head workgroups:
//   coarse gates of all units (every head, redundantly)
//   -> own O1 rows + O2 columns -> partial coarse logits   --hop-->  all heads
//   -> sum, draw c_t (every head, identically) -> fine gates of all units
//   -> own O3 rows + O4 columns -> partial fine logits, and own rows of
//      R_c[:, fine] y_f (the part of the next coarse pre-activation that
//      depends on y_f)                                      --hop-->  all heads
//   -> sum, draw f_t -> next step.
// Off the critical path, NU unit workgroups receive y_c and y_f and compute the
// rest of R h (coarse rows x coarse inputs, fine rows x all inputs), adding the
// gate bias and conditioning, one step ahead of when the heads need them.
#include "wr_device.h"
#include "wr_layout.h"
#include "wr_args.h"

// ---------------------------------------------------------------------------
// Arithmetic of this kernel: hardware exp2 / reciprocal (about 1 ulp).  The
// single-workgroup kernel keeps the exactly specified functions instead.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float fsig(float x) { return frcp(1.0f + fexp(-x)); }
__device__ __forceinline__ float ftanh(float x) {
  float q = fexp(-2.0f * __builtin_fabsf(x));
  return __builtin_copysignf((1.0f - q) * frcp(1.0f + q), x);
}
__device__ __forceinline__ float fscale(int v) { return (float)(2 * v - 255) * (1.0f / 255.0f); }

// DPP cross-lane moves (wave64, gfx9 row_shr / row_bcast / wave_shr).
template <int CTRL, int ROWMASK, bool BOUND_ZERO>
__device__ __forceinline__ float dpp(float old, float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), CTRL, ROWMASK, 0xf, BOUND_ZERO));
}
__device__ __forceinline__ float lane63(float v) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63)); }

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ float wave_scan(float v) {
  v += dpp<0x111, 0xf, true>(0.0f, v);   // row_shr:1
  v += dpp<0x112, 0xf, true>(0.0f, v);   // row_shr:2
  v += dpp<0x114, 0xf, true>(0.0f, v);   // row_shr:4
  v += dpp<0x118, 0xf, true>(0.0f, v);   // row_shr:8
  v += dpp<0x142, 0xa, false>(0.0f, v);  // row_bcast:15 -> rows 1, 3
  v += dpp<0x143, 0xc, false>(0.0f, v);  // row_bcast:31 -> rows 2, 3
  return v;
}
// Maximum over the 64 lanes (uniform result).
__device__ __forceinline__ float wave_maxf(float v) {
  const float NI = -__builtin_inff();
  v = fmaxf(v, dpp<0x111, 0xf, false>(NI, v));
  v = fmaxf(v, dpp<0x112, 0xf, false>(NI, v));
  v = fmaxf(v, dpp<0x114, 0xf, false>(NI, v));
  v = fmaxf(v, dpp<0x118, 0xf, false>(NI, v));
  v = fmaxf(v, dpp<0x142, 0xa, false>(NI, v));
  v = fmaxf(v, dpp<0x143, 0xc, false>(NI, v));
  return lane63(v);
}

// Inverse-CDF draw over softmax(z) by one wave, 4 classes per lane (z in LDS).
// Returns the class, or `forced` when >= 0; *lse = max z + log sum exp(z - max).
__device__ int draw_wave(const float* z, float u, int forced, float* lse) {
  const int l = threadIdx.x & 63;
  float4 z4 = *(const float4*)(z + 4 * l);
  float m = wave_maxf(fmaxf(fmaxf(z4.x, z4.y), fmaxf(z4.z, z4.w)));
  float w0 = fexp(z4.x - m), w1 = fexp(z4.y - m), w2 = fexp(z4.z - m), w3 = fexp(z4.w - m);
  float s0 = w0, s1 = s0 + w1, s2 = s1 + w2, s3 = s2 + w3;
  float incl = wave_scan(s3);
  float excl = dpp<0x138, 0xf, true>(0.0f, incl);   // wave_shr:1, lane 0 gets 0
  float Z = lane63(incl);
  if (lse) *lse = m + __logf(Z);
  if (forced >= 0) return forced;
  float thr = u * Z;
  int count = __popcll(__ballot(excl + s0 <= thr)) + __popcll(__ballot(excl + s1 <= thr)) +
              __popcll(__ballot(excl + s2 <= thr)) + __popcll(__ballot(excl + s3 <= thr));
  if (count == WR_CLASSES) {   // clamp to the last class with nonzero weight
    int last = -1;
    u64 b;
    if ((b = __ballot(w3 > 0.0f))) last = max(last, 4 * (63 - __clzll(b)) + 3);
    if ((b = __ballot(w2 > 0.0f))) last = max(last, 4 * (63 - __clzll(b)) + 2);
    if ((b = __ballot(w1 > 0.0f))) last = max(last, 4 * (63 - __clzll(b)) + 1);
    if ((b = __ballot(w0 > 0.0f))) last = max(last, 4 * (63 - __clzll(b)));
    count = last;
  }
  return count;
}

// ---------------------------------------------------------------------------
// Matrix-vector products on the matrix cores.  v_mfma_f32_16x16x32_bf16 with
// the vector as operand A: row 0 holds the bf16 high part of x, row 1 the bf16
// low part (x - high, rounded), rows 2..15 are zero; the weights are operand B
// (see the fragment layout in wr_layout.h).  Products of bf16 values are exact
// in fp32, so W x is carried to about 2^-16 relative per term, and lanes 0..15
// of the result hold the 16 output rows of the tile: D[0][n] + D[1][n].
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Operand-A fragment of x[32*kt .. 32*kt+31] (x fp32 in LDS).  Every lane reads
// its 8 values (no divergence); lanes of rows >= 2 contribute zeros.
__device__ __forceinline__ bf16x8 xfrag(const float* x, int kt) {
  const int l = threadIdx.x & 63, r = l & 15, kq = l >> 4;
  const float* src = x + 32 * kt + 8 * kq;
  float4 a = *(const float4*)src, b = *(const float4*)(src + 4);
  float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float hi = __uint_as_float(__float_as_uint(v[i]) & 0xffff0000u);
    float sel = r == 0 ? hi : (r == 1 ? v[i] - hi : 0.0f);
    f[i] = (__bf16)sel;
  }
  return f;
}

__device__ __forceinline__ bf16x8 wfrag(const unsigned char* base, int idx) {
  return *(const bf16x8*)(base + ((size_t)idx * 64 + (threadIdx.x & 63)) * 16);
}

// Partial products of row tiles m0 .. m0+MT-1 over column tiles kt = k0, k0+ks,
// ... < KT (x covers all KT tiles; the matrix has KT column tiles per row tile).
// The MT weight fragments of a column tile are read together before its MFMAs.
// out[16*m + n] receives row 16*(m0+m) + n from lane n.
template <int MT>
__device__ __forceinline__ void tile_rows(const unsigned char* W, int KT, const float* x, int m0, int k0, int ks,
                                          float* out) {
  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  for (int kt = k0; kt < KT; kt += ks) {
    bf16x8 wc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) wc[m] = wfrag(W, (m0 + m) * KT + kt);
    const bf16x8 xa = xfrag(x, kt);
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = mfma(xa, wc[m], acc[m]);
  }
  const int l = threadIdx.x & 63;
  if (l < 16) {
#pragma unroll
    for (int m = 0; m < MT; ++m) out[16 * m + l] = acc[m][0] + acc[m][1];
  }
}

// Wait until every word p[k] (k < N) carries `tag`, with all loads of a round in
// flight together; false on timeout / abort.
template <int N>
__device__ __forceinline__ bool poll_n(const u64* const* p, uint32_t tag, float* v, WaitBudget& wb,
                                       const PersistArgs& a) {
  uint32_t pending = (1u << N) - 1u;
  for (;;) {
    u64 w[N];
#pragma unroll
    for (int k = 0; k < N; ++k) w[k] = (pending >> k & 1u) ? xpeek(p[k]) : 0;
#pragma unroll
    for (int k = 0; k < N; ++k)
      if ((pending >> k & 1u) && xtag(w[k]) == tag) {
        v[k] = xval(w[k]);
        pending &= ~(1u << k);
      }
    if (!pending) return true;
    if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
}

// Like poll_n, starting from words w[] loaded earlier (prefetched): only the
// words that did not yet carry `tag` are loaded again.
template <int N>
__device__ __forceinline__ bool poll_pref(const u64* const* p, const u64* w, uint32_t tag, float* v, WaitBudget& wb,
                                          const PersistArgs& a) {
  uint32_t pending = 0;
#pragma unroll
  for (int k = 0; k < N; ++k) {
    if (xtag(w[k]) == tag) v[k] = xval(w[k]);
    else pending |= 1u << k;
  }
  while (pending) {
    u64 x[N];
#pragma unroll
    for (int k = 0; k < N; ++k) x[k] = (pending >> k & 1u) ? xpeek(p[k]) : 0;
#pragma unroll
    for (int k = 0; k < N; ++k)
      if ((pending >> k & 1u) && xtag(x[k]) == tag) {
        v[k] = xval(x[k]);
        pending &= ~(1u << k);
      }
    if (pending && !wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
  return true;
}

// Wait until *p carries `tag`; false on timeout / abort.
__device__ __forceinline__ bool poll1(const u64* p, uint32_t tag, float* v, WaitBudget& wb, const PersistArgs& a) {
  u64 w;
  while (xtag(w = xpeek(p)) != tag)
    if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
  *v = xval(w);
  return true;
}

// Gather n tagged words into dst (all threads, up to 2 words each).
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

// Sum of partial logits p[j*256 + v] for parts j in [j0, j0 + np) in part
// order, once all carry `tag` (all pending words of a round loaded together).
template <int MAXP>
__device__ bool sum_parts(const u64* src, int j0, int np, int v, uint32_t tag, float* out, const PersistArgs& a) {
  WaitBudget wb{wr_clock(), 0};
  float vals[MAXP];
  uint32_t pending = (1u << np) - 1u;
  while (pending) {
    u64 w[MAXP];
#pragma unroll
    for (int k = 0; k < MAXP; ++k) w[k] = (pending >> k & 1u) ? xpeek(src + (j0 + k) * WR_CLASSES + v) : 0;
#pragma unroll
    for (int k = 0; k < MAXP; ++k)
      if ((pending >> k & 1u) && xtag(w[k]) == tag) {
        vals[k] = xval(w[k]);
        pending &= ~(1u << k);
      }
    if (pending && !wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
  float acc = 0.0f;
#pragma unroll
  for (int k = 0; k < MAXP; ++k)
    if (k < np) acc += vals[k];
  *out = acc;
  return true;
}

// Phase timestamp of a traced step.
__device__ __forceinline__ void trace_at(const PersistArgs& a, int64_t t, int slot) {
  if (a.trace && t < a.trace_steps) a.trace[t * WR_TRACE_SLOTS + slot] = wr_clock();
}

// Bias + conditioning of R row `row` for absolute sample n.
__device__ float gate_add(const PersistArgs& a, int row, int64_t n) {
  float v = a.bias[row];
  if (a.Dc > 0) {
    int64_t fr = n / a.frame_len;
    if (fr >= a.n_frames) fr = a.n_frames - 1;
    const float* wc = a.Wc + (size_t)row * a.Dc;
    const float* fv = a.feat + (size_t)fr * a.Dc;
    float acc = 0.0f;
    for (int q = 0; q < a.Dc; ++q) acc = __builtin_fmaf(wc[q], fv[q], acc);
    v = acc + v;
  }
  return v;
}

// ------------------------------------------------------------------ head role
__device__ void head_role(const PersistArgs& a, int j, unsigned char* lds) {
  const PersistPlan& P = a.P;
  const int H = P.H, Hh = P.Hh, NH = P.NH, KT = P.KT;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const unsigned char* W1 = lds + P.hb_o1;
  const unsigned char* W3 = lds + P.hb_o3;
  const unsigned char* WR = lds + P.hb_rcf;
  float* h = (float*)(lds + P.h_bytes);  // [H] hidden state (identical in every head)
  float* z = h + H;                      // [256] logits
  float* zh = z + 256;                   // [256] second half of the partial-logit sums
  float* op = zh + 256;                  // [8][32] first-layer partials per wave
  float* rp = op + 8 * WR_HR;            // [4][96] R_c[:, fine] y_f partials per wave
  float* ov = rp + 4 * WR_GR;            // [32] relu(first layer) of this head's rows
  float* bs = ov + WR_HR;                // [0:32] b1 slice, [32:64] b3 slice
  int* misc = (int*)(bs + 64);           // [0] abort [1] c_t [3] c_prev [4] f_prev
  float* fmisc = (float*)(misc + 8);     // [0] u_c [1] u_f [2] lse_c [3] z_c[c]

  // --- prologue
  {
    const uint4* src = a.wh + (size_t)j * (P.h_bytes / 16);
    uint4* dst = (uint4*)lds;
    for (int i = tid; i < P.h_bytes / 16; i += blockDim.x) dst[i] = src[i];
    for (int i = tid; i < H; i += blockDim.x) h[i] = a.h_in ? a.h_in[i] : 0.0f;
    if (tid < WR_HR) {
      bs[tid] = a.b1[j * WR_HR + tid];
      bs[WR_HR + tid] = a.b3[j * WR_HR + tid];
    }
    if (tid == 0) {
      misc[0] = 0;
      misc[3] = a.c_in ? a.c_in[0] : 128;
      misc[4] = a.f_in ? a.f_in[0] : 0;
    }
  }
  // O2 / O4 column-slice fragments of class tiles 4*wave .. 4*wave+3 (waves 0-3)
  bf16x8 o2f[4], o4f[4];
  if (wave < 4) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 x2 = a.o2s[((size_t)j * 16 + 4 * wave + s) * 64 + lane];
      uint4 x4 = a.o4s[((size_t)j * 16 + 4 * wave + s) * 64 + lane];
      o2f[s] = __builtin_bit_cast(bf16x8, x2);
      o4f[s] = __builtin_bit_cast(bf16x8, x4);
    }
  }
  // I* rows of unit u = tid: coarse (c_{t-1}, f_{t-1}), fine (c_{t-1}, f_{t-1}, c_t)
  float ic[3][2], ifn[3][3];
  const int u = tid;
  if (u < Hh) {
#pragma unroll
    for (int g = 0; g < 3; ++g) {
      ic[g][0] = a.Iw[3 * (g * H + u) + 0];
      ic[g][1] = a.Iw[3 * (g * H + u) + 1];
      ifn[g][0] = a.Iw[3 * (g * H + Hh + u) + 0];
      ifn[g][1] = a.Iw[3 * (g * H + Hh + u) + 1];
      ifn[g][2] = a.Iw[3 * (g * H + Hh + u) + 2];
    }
  }
  const float b2v = tid < WR_CLASSES ? a.b2[tid] : 0.0f;
  const float b4v = tid < WR_CLASSES ? a.b4[tid] : 0.0f;
  __syncthreads();

  const u64* GA = a.xc + P.x_ga;
  const u64* GF = a.xc + P.x_gf;
  u64* GCF = a.xc + P.x_gcf;
  const u64* AEC = a.xc + P.x_aec;
  const u64* AEF = a.xc + P.x_aef;
  u64* YC = a.xc + P.x_yc;
  u64* YF = a.xc + P.x_yf;
  u64* PCo = a.xc + P.x_pc + (size_t)j * WR_CLASSES;
  u64* PFo = a.xc + P.x_pf + (size_t)j * WR_CLASSES;
  const u64* PC = a.xc + P.x_pc;
  const u64* PF = a.xc + P.x_pf;

  // R_c[:, fine] y_f partials of this head's rows on waves 4-7, summed by
  // threads 256..351 after a barrier and published with `tag`.
  // wave 4 + 2*kh + mh: row tiles 3*mh .. 3*mh+2, column tiles kh, kh+2, ...
  auto rcf_partial = [&]() {
    const int w4 = wave - 4, mh = w4 & 1, kh = w4 >> 1;
    tile_rows<WR_GR / 32>(WR, KT, h + Hh, 3 * mh, kh, 2, rp + kh * WR_GR + mh * (WR_GR / 2));
  };
  auto rcf_publish = [&](uint32_t tag) {
    const int r = tid - 256;
    if (r >= 0 && r < WR_GR) xpub(GCF + j * WR_GR + r, tag, rp[r] + rp[WR_GR + r]);
  };
  // relu(first layer + bias) of this head's rows from nparts wave partials
  auto relu_rows = [&](int nparts, const float* b) {
    if (tid < WR_HR) {
      float s = 0.0f;
      for (int w = 0; w < nparts; ++w) s += op[w * WR_HR + tid];
      ov[tid] = wr_relu(s + b[tid]);
    }
  };
  // second layer on waves 0-3: partial logits of class tiles 4*wave .. +3
  auto second_layer = [&](const bf16x8* of, u64* dst, uint32_t tag) {
    const bf16x8 xa = xfrag(ov, 0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      f32x4 acc = mfma(xa, of[s], f32x4{0.0f, 0.0f, 0.0f, 0.0f});
      if (lane < 16) xpub(dst + 16 * (4 * wave + s) + lane, tag, acc[0] + acc[1]);
    }
  };

  // step 0's R_c[:, fine] y_f(-1) from the initial state
  if (wave >= 4) rcf_partial();
  __syncthreads();
  rcf_publish(1u);

  // prefetched pre-activation words of this thread's unit: coarse (GA x3,
  // GCF x3, AEC) and fine (GF x3, AEF); loaded a phase before they are needed
  u64 pc7[7] = {0, 0, 0, 0, 0, 0, 0}, pf4[4] = {0, 0, 0, 0};
  auto prefetch_coarse = [&]() {
    if (u < Hh) {
      pc7[0] = xpeek(GA + u); pc7[1] = xpeek(GA + Hh + u); pc7[2] = xpeek(GA + 2 * Hh + u);
      pc7[3] = xpeek(GCF + u); pc7[4] = xpeek(GCF + Hh + u); pc7[5] = xpeek(GCF + 2 * Hh + u);
      pc7[6] = xpeek(AEC + u);
    }
  };
  auto prefetch_fine = [&]() {
    if (u < Hh) {
      pf4[0] = xpeek(GF + u); pf4[1] = xpeek(GF + Hh + u); pf4[2] = xpeek(GF + 2 * Hh + u);
      pf4[3] = xpeek(AEF + u);
    }
  };
  const int half_parts = (NH + 1) / 2;

  for (int64_t t = 0; t < a.T; ++t) {
    const int64_t n = a.t0 + t;
    const uint32_t tag = (uint32_t)(t + 1);
    const bool tr = j == 0 && tid == 0;
    const bool trl = j == NH - 1 && j > 0 && tid == 0;   // last head: fine partials published
    if (tr) trace_at(a, t, 0);
    if (tid == 64) {
      float uc, uf;
      wr_uniforms(a.seed, a.stream_id, (uint64_t)n, &uc, &uf);
      fmisc[0] = uc;
      fmisc[1] = uf;
    }
    // (1)-(2) coarse gates of every unit
    const float x0 = fscale(misc[3]), x1 = fscale(misc[4]);
    bool ok = true;
    if (u < Hh) {
      WaitBudget wb{wr_clock(), 0};
      const u64* ps[7] = {GA + u, GA + Hh + u, GA + 2 * Hh + u, GCF + u, GCF + Hh + u, GCF + 2 * Hh + u, AEC + u};
      float v[7];
      ok = poll_pref<7>(ps, pc7, tag, v, wb, a);
      if (ok) {
        float au = (v[0] + v[3]) + __builtin_fmaf(ic[0][1], x1, ic[0][0] * x0);
        float ar = (v[1] + v[4]) + __builtin_fmaf(ic[1][1], x1, ic[1][0] * x0);
        float ie = __builtin_fmaf(ic[2][1], x1, ic[2][0] * x0) + v[6];
        float uu = fsig(au), rr = fsig(ar);
        float e = ftanh(__builtin_fmaf(rr, v[2] + v[5], ie));
        float hn = __builtin_fmaf(uu, h[u], (1.0f - uu) * e);
        h[u] = hn;
        if (u >= j * WR_HR && u < (j + 1) * WR_HR) xpub(YC + u, tag, hn);
      }
    }
    if (!ok) misc[0] = 1;
    __syncthreads();
    if (misc[0]) return;
    if (tr) trace_at(a, t, 1);
    // (3) O1 rows of this head: column tiles split over the 8 waves
    tile_rows<WR_HR / 16>(W1, KT, h, 0, wave, 8, op + wave * WR_HR);
    if (tr) trace_at(a, t, 18);
    __syncthreads();
    if (tr) trace_at(a, t, 19);
    relu_rows(8, bs);
    __syncthreads();
    if (tr) trace_at(a, t, 2);
    // (4) partial coarse logits
    if (wave < 4) second_layer(o2f, PCo, tag);
    if (tr) trace_at(a, t, 3);

    // (5) sum partials of all heads (two threads per class), fine words prefetched
    prefetch_fine();
    {
      const int v = tid & 255, hf = tid >> 8;
      float s;
      if (!sum_parts<(WR_MAXNH + 1) / 2>(PC, hf ? half_parts : 0, hf ? NH - half_parts : half_parts, v, tag, &s, a))
        misc[0] = 1;
      else if (hf) zh[v] = s;
      else z[v] = s;
    }
    __syncthreads();
    if (misc[0]) return;
    if (tid < WR_CLASSES) z[tid] = (z[tid] + zh[tid]) + b2v;
    __syncthreads();
    if (tr) trace_at(a, t, 4);
    // (6) draw c_t (every head draws the same class)
    const int64_t o = t;
    if (j == 0 && a.zc_out && tid < WR_CLASSES) a.zc_out[o * WR_CLASSES + tid] = z[tid];
    if (wave == 0) {
      float lse;
      int forced = a.target ? (a.target[o] >> 8) : -1;
      int c = draw_wave(z, fmisc[0], forced, a.nll_out ? &lse : nullptr);
      if (lane == 0) {
        misc[1] = c;
        if (a.nll_out) {
          fmisc[2] = lse;
          fmisc[3] = z[c];
        }
      }
    }
    __syncthreads();
    if (tr) trace_at(a, t, 5);
    // (7)-(8) fine gates of every unit (c_t reaches the fine half only)
    const int c = misc[1];
    if (u < Hh) {
      WaitBudget wb{wr_clock(), 0};
      const u64* ps[4] = {GF + u, GF + Hh + u, GF + 2 * Hh + u, AEF + u};
      float v[4];
      ok = poll_pref<4>(ps, pf4, tag, v, wb, a);
      if (ok) {
        const float x2 = fscale(c);
        float au = v[0] + __builtin_fmaf(ifn[0][2], x2, __builtin_fmaf(ifn[0][1], x1, ifn[0][0] * x0));
        float ar = v[1] + __builtin_fmaf(ifn[1][2], x2, __builtin_fmaf(ifn[1][1], x1, ifn[1][0] * x0));
        float ie = __builtin_fmaf(ifn[2][2], x2, __builtin_fmaf(ifn[2][1], x1, ifn[2][0] * x0)) + v[3];
        float uu = fsig(au), rr = fsig(ar);
        float e = ftanh(__builtin_fmaf(rr, v[2], ie));
        float hn = __builtin_fmaf(uu, h[Hh + u], (1.0f - uu) * e);
        h[Hh + u] = hn;
        if (u >= j * WR_HR && u < (j + 1) * WR_HR) xpub(YF + u, tag, hn);
      }
    }
    if (!ok) misc[0] = 1;
    __syncthreads();
    if (misc[0]) return;
    if (tr) trace_at(a, t, 6);
    // (9)-(10) O3 rows on waves 0-3, this head's rows of R_c[:, fine] y_f(t) on waves 4-7
    if (wave < 4) tile_rows<WR_HR / 16>(W3, KT, h + Hh, 0, wave, 4, op + wave * WR_HR);
    else if (t + 1 < a.T) rcf_partial();
    if (tr) trace_at(a, t, 12);
    if (j == 0 && tid == 256) trace_at(a, t, 13);
    __syncthreads();
    if (tr) trace_at(a, t, 14);
    relu_rows(4, bs + WR_HR);
    if (t + 1 < a.T) rcf_publish(tag + 1);
    if (j == 0 && tid == 256) trace_at(a, t, 15);
    __syncthreads();
    if (tr) trace_at(a, t, 16);
    if (wave < 4) second_layer(o4f, PFo, tag);
    if (tr) trace_at(a, t, 17);
    if (tr) trace_at(a, t, 7);
    if (trl) trace_at(a, t, 11);
    // (11) sum partials, draw f_t; next step's coarse words prefetched
    prefetch_coarse();
    {
      const int v = tid & 255, hf = tid >> 8;
      float s;
      if (!sum_parts<(WR_MAXNH + 1) / 2>(PF, hf ? half_parts : 0, hf ? NH - half_parts : half_parts, v, tag, &s, a))
        misc[0] = 1;
      else if (hf) zh[v] = s;
      else z[v] = s;
    }
    __syncthreads();
    if (misc[0]) return;
    if (tid < WR_CLASSES) z[tid] = (z[tid] + zh[tid]) + b4v;
    __syncthreads();
    if (tr) trace_at(a, t, 9);
    if (j == 0 && a.zf_out && tid < WR_CLASSES) a.zf_out[o * WR_CLASSES + tid] = z[tid];
    if (wave == 0) {
      float lse;
      int forced = a.target ? (a.target[o] & 255) : -1;
      int f = draw_wave(z, fmisc[1], forced, a.nll_out ? &lse : nullptr);
      if (lane == 0) {
        if (j == 0) {
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
  if (j == 0) {
    if (a.h_out)
      for (int i = tid; i < H; i += blockDim.x) a.h_out[i] = h[i];
    if (tid == 0) {
      if (a.c_out) a.c_out[0] = (uint8_t)misc[3];
      if (a.f_out) a.f_out[0] = (uint8_t)misc[4];
    }
  }
}

// ------------------------------------------------------------------ unit role
// GA rows cr = k*UR + m (coarse rows x coarse inputs) and GF rows fr = k*UR + m
// (fine rows x both inputs), m < UR; column tiles split over the 8 waves.
// Bias + conditioning is added for gates u and r; for gate e it is published
// separately (AEC / AEF) because the reset gate multiplies R_e h only.
__device__ void unit_role(const PersistArgs& a, int k, unsigned char* lds) {
  const PersistPlan& P = a.P;
  const int H = P.H, Hh = P.Hh, KT = P.KT;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const unsigned char* WGA = lds + P.ub_ga;
  const unsigned char* WGF = lds + P.ub_gf;
  float* y = (float*)(lds + P.u_bytes);  // [H]
  float* gp = y + H;                     // [8][UR] GA partials
  float* fp = gp + 8 * WR_UR;            // [8][UR] GF partials
  int* misc = (int*)(fp + 8 * WR_UR);
  {
    const uint4* src = a.wu + (size_t)k * (P.u_bytes / 16);
    uint4* dst = (uint4*)lds;
    for (int i = tid; i < P.u_bytes / 16; i += blockDim.x) dst[i] = src[i];
    for (int i = tid; i < H; i += blockDim.x) y[i] = a.h_in ? a.h_in[i] : 0.0f;
    if (tid == 0) misc[0] = 0;
  }
  // row of this thread for the publish phases: tid < UR -> GA row, 64 <= tid < 64+UR -> GF row
  const bool pub_ga = tid < WR_UR, pub_gf = tid >= 64 && tid < 64 + WR_UR;
  const int m = pub_ga ? tid : tid - 64;
  const int xr = k * WR_UR + m;            // row index within its half, g*Hh + i
  const int g = xr / Hh, i = xr % Hh;
  const int grow = pub_ga ? g * H + i : g * H + Hh + i;
  int64_t cur_frame = -2;
  float addr = 0.0f;
  auto refresh_add = [&](int64_t n) {      // bias + conditioning of this thread's row for sample n
    int64_t fr = a.Dc > 0 ? n / a.frame_len : 0;
    if (fr != cur_frame) {
      cur_frame = fr;
      if (pub_ga || pub_gf) addr = gate_add(a, grow, n);
    }
  };
  auto publish = [&](uint32_t tag, const float* part) {
    if (!(pub_ga || pub_gf)) return;
    float acc = 0.0f;
    for (int w = 0; w < 8; ++w) acc += part[w * WR_UR + m];
    u64* dst = a.xc + (pub_ga ? P.x_ga : P.x_gf) + xr;
    if (g == 2) {
      xpub(dst, tag, acc);
      xpub(a.xc + (pub_ga ? P.x_aec : P.x_aef) + i, tag, addr);
    } else {
      xpub(dst, tag, acc + addr);
    }
  };
  // GF rows accumulate over both input halves: column tiles 0..KT-1 (y_c) then KT..2KT-1 (y_f)
  f32x4 gfa[WR_UR / 16];
  auto gf_tiles = [&](int k0, int k1) {
    for (int kt = k0 + ((wave - k0) % 8 + 8) % 8; kt < k1; kt += 8) {
      bf16x8 wc[WR_UR / 16];
#pragma unroll
      for (int mt = 0; mt < WR_UR / 16; ++mt) wc[mt] = wfrag(WGF, mt * 2 * KT + kt);
      const bf16x8 xa = xfrag(y, kt);
#pragma unroll
      for (int mt = 0; mt < WR_UR / 16; ++mt) gfa[mt] = mfma(xa, wc[mt], gfa[mt]);
    }
  };
  auto gf_store = [&]() {
    if (lane < 16) {
#pragma unroll
      for (int mt = 0; mt < WR_UR / 16; ++mt) fp[wave * WR_UR + 16 * mt + lane] = gfa[mt][0] + gfa[mt][1];
    }
  };
  __syncthreads();
  // step 0's pre-activations from the initial state
  refresh_add(a.t0);
  tile_rows<WR_UR / 16>(WGA, KT, y, 0, wave, 8, gp + wave * WR_UR);
#pragma unroll
  for (int mt = 0; mt < WR_UR / 16; ++mt) gfa[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  gf_tiles(0, 2 * KT);
  gf_store();
  __syncthreads();
  publish(1u, pub_ga ? gp : fp);
  const u64* YC = a.xc + P.x_yc;
  const u64* YF = a.xc + P.x_yf;
  for (int64_t t = 0; t + 1 < a.T; ++t) {
    const uint32_t tag = (uint32_t)(t + 1), ntag = tag + 1;
    refresh_add(a.t0 + t + 1);
    if (!gather_words(YC, Hh, tag, y, a)) misc[0] = 1;
    __syncthreads();
    if (misc[0]) return;
    tile_rows<WR_UR / 16>(WGA, KT, y, 0, wave, 8, gp + wave * WR_UR);
#pragma unroll
    for (int mt = 0; mt < WR_UR / 16; ++mt) gfa[mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    gf_tiles(0, KT);
    __syncthreads();
    if (pub_ga) publish(ntag, gp);
    if (!gather_words(YF, Hh, tag, y + Hh, a)) misc[0] = 1;
    __syncthreads();
    if (misc[0]) return;
    gf_tiles(KT, 2 * KT);
    gf_store();
    __syncthreads();
    if (pub_gf) publish(ntag, fp);
  }
}

extern "C" __global__ __launch_bounds__(WR_THREADS, 1) void wr_persist_kernel(PersistArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int b = blockIdx.x;
  if (b < a.P.NH) head_role(a, b, lds);
  else unit_role(a, b - a.P.NH, lds);
}

extern "C" __global__ void wr_fill_u64(u64* p, int64_t n, u64 v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

const void* wr_persist_kernel_ptr() { return (const void*)wr_persist_kernel; }

const void* wr_fill_kernel_ptr() { return (const void*)wr_fill_u64; }
