// Device building blocks shared by the persistent kernels of libwavernn
// (fast elementwise functions, wave-level scans and the inverse-CDF draw,
// matrix-core matrix-vector fragments, bounded waits on tagged words).
#pragma once
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

// Inverse-CDF draw by one wave over z = p + b, classes 4 l .. 4 l + 3 on lane
// l.  The logits are also written to zkeep[256].  Returns the class, or
// `forced` when >= 0; *lse = max z + log sum exp(z - max).
__device__ __forceinline__ int draw_z(float4 p, float4 b, float u, int forced, float* zkeep, float* lse) {
  const int l = threadIdx.x & 63;
  float4 z4;
  z4.x = p.x + b.x;
  z4.y = p.y + b.y;
  z4.z = p.z + b.z;
  z4.w = p.w + b.w;
  *(float4*)(zkeep + 4 * l) = z4;
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
    u64 bb;
    if ((bb = __ballot(w3 > 0.0f))) last = max(last, 4 * (63 - __clzll(bb)) + 3);
    if ((bb = __ballot(w2 > 0.0f))) last = max(last, 4 * (63 - __clzll(bb)) + 2);
    if ((bb = __ballot(w1 > 0.0f))) last = max(last, 4 * (63 - __clzll(bb)) + 1);
    if ((bb = __ballot(w0 > 0.0f))) last = max(last, 4 * (63 - __clzll(bb)));
    count = last;
  }
  return count;
}
// draw_z over p = zs + zs2 (zs alone when !TWO), read from LDS.
template <bool TWO = true>
__device__ __forceinline__ int draw_wave(const float* zs, const float* zs2, float4 b, float u, int forced,
                                         float* zkeep, float* lse) {
  const int l = threadIdx.x & 63;
  float4 p = *(const float4*)(zs + 4 * l);
  if (TWO) {
    const float4 q = *(const float4*)(zs2 + 4 * l);
    p.x += q.x;
    p.y += q.y;
    p.z += q.z;
    p.w += q.w;
  }
  return draw_z(p, b, u, forced, zkeep, lse);
}

// ---------------------------------------------------------------------------
// Matrix-vector products on the matrix cores.  v_mfma_f32_16x16x32_bf16 with
// the vector as operand A: row 0 holds the bf16 high part of x, row 1 the bf16
// low part (x - high, rounded), rows 2..15 are zero; the weights are operand B
// (fragment layout in wr_layout.h).  Products of bf16 values are exact in
// fp32, so W x is carried to about 2^-16 relative per term, and lane n < 16 of
// the result holds output row n of the tile as D[0][n] + D[1][n].
//
// The operand-A images live in LDS in fragment order (1 KiB per 32 inputs,
// lane l's 16 bytes at 16 l), rows 2..15 zeroed once: writing input k of a
// tile sets two bf16 values, and every lane reads its operand with one
// 16-byte LDS load.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8 afrag(const unsigned char* img, int kt) {
  return *(const bf16x8*)(img + kt * WR_FRAG + (threadIdx.x & 63) * 16);
}
// Store x as input k (0 <= k < 32) of operand tile `img`, rows 2b and 2b+1
// (vector b of a batch; a single vector uses rows 0 and 1).
__device__ __forceinline__ void aput(unsigned char* img, int k, float x, int b = 0) {
  const float hi = __uint_as_float(__float_as_uint(x) & 0xffff0000u);
  const __bf16 bh = (__bf16)hi, bl = (__bf16)(x - hi);
  __bf16* row0 = (__bf16*)(img + (16 * (k >> 3) + 2 * b) * 16) + (k & 7);
  row0[0] = bh;        // lane 16*(k/8) + 2b,     element k%8
  row0[8] = bl;        // lane 16*(k/8) + 2b + 1, element k%8
}
// Output row n of a tile for vector 0 (lane n < 16), or for vectors 2(l/16) and
// 2(l/16) + 1 of a batch (every lane l holds rows 4(l/16) .. 4(l/16)+3).
__device__ __forceinline__ float mfma_row(f32x4 d) { return d[0] + d[1]; }
__device__ __forceinline__ float mfma_row_hi(f32x4 d) { return d[2] + d[3]; }

// ---------------------------------------------------------------------------
// Waits on tagged words (bounded: see WaitBudget).
// ---------------------------------------------------------------------------
// Wait until every word p[k] (k < N) carries `tag`, starting from words w[]
// loaded earlier; only words that did not carry it yet are loaded again.
template <int N, class A>
__device__ __forceinline__ bool poll_pref(const xw* const* p, const xw* w, uint32_t tag, float* v, const A& a) {
  uint32_t pending = 0;
#pragma unroll
  for (int k = 0; k < N; ++k) {
    if (xok(w[k], tag)) v[k] = xval(w[k]);
    else pending |= 1u << k;
  }
  if (!pending) return true;
  WaitBudget wb{wr_clock(), 0};
  while (pending) {
    xw x[N];
#pragma unroll
    for (int k = 0; k < N; ++k) x[k] = (pending >> k & 1u) ? xpeek(p[k]) : 0;
#pragma unroll
    for (int k = 0; k < N; ++k)
      if ((pending >> k & 1u) && xok(x[k], tag)) {
        v[k] = xval(x[k]);
        pending &= ~(1u << k);
      }
    if (pending && !wait_ok(wb, a.err, a.limit, a.err)) return false;
  }
  return true;
}

// Wait until *p carries `tag` (with SLEEP, a short sleep between loads).
template <bool SLEEP = true, class A>
__device__ __forceinline__ bool poll_sleepy(const xw* p, uint32_t tag, float* v, const A& a) {
  xw w = xpeek(p);
  if (!xok(w, tag)) {
    WaitBudget wb{wr_clock(), 0};
    do {
      if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
      if (SLEEP) __builtin_amdgcn_s_sleep(1);
    } while (!xok(w = xpeek(p), tag));
  }
  *v = xval(w);
  return true;
}

// Sum over parts jj = j0 .. j1-1 of src[jj*stride + v] once all carry `tag`, in
// part order (every head sums in the same order, so all draw the same class).
template <int MAXP, class A>
__device__ __forceinline__ bool sum_parts(const xw* src, int stride, int j0, int j1, int v, uint32_t tag, float* out,
                                          const A& a) {
  float vals[MAXP];
  uint32_t pending = 0;
  xw w[MAXP];
#pragma unroll
  for (int k = 0; k < MAXP; ++k) w[k] = j0 + k < j1 ? xpeek(src + (size_t)(j0 + k) * stride + v) : 0;
#pragma unroll
  for (int k = 0; k < MAXP; ++k) {
    if (j0 + k >= j1) continue;
    if (xok(w[k], tag)) vals[k] = xval(w[k]);
    else pending |= 1u << k;
  }
  if (pending) {
    WaitBudget wb{wr_clock(), 0};
    while (pending) {
      if (!wait_ok(wb, a.err, a.limit, a.err)) return false;
#pragma unroll
      for (int k = 0; k < MAXP; ++k) w[k] = (pending >> k & 1u) ? xpeek(src + (size_t)(j0 + k) * stride + v) : 0;
#pragma unroll
      for (int k = 0; k < MAXP; ++k)
        if ((pending >> k & 1u) && xok(w[k], tag)) {
          vals[k] = xval(w[k]);
          pending &= ~(1u << k);
        }
    }
  }
  float acc = 0.0f;
#pragma unroll
  for (int k = 0; k < MAXP; ++k)
    if (j0 + k < j1) acc += vals[k];
  *out = acc;
  return true;
}

// Phase timestamp of a traced step.
template <class A>
__device__ __forceinline__ void trace_at(const A& a, int64_t t, int slot) {
  if (a.trace && t < a.trace_steps) a.trace[t * WR_TRACE_SLOTS + slot] = wr_clock();
}

// Words that only the lead workgroups read (partial logits, the mirrors'
// words) are published into the L2 of their XCD when all leads share one
// (build with WR_LOCAL_XCHG=0 to keep every word coherent across XCDs).
#ifndef WR_LOCAL_XCHG
#define WR_LOCAL_XCHG 1
#endif
// Do all n lead workgroups of a launch (the heads and mirrors of a batch-1
// grid, placed on one XCD) run on one XCD?  Lead i publishes its XCD (the
// XCC_ID hardware register) in words[i] and thread 0 reads every lead's; all
// leads read the same words, so all get the same answer.  Called by every
// thread of the workgroup (one barrier inside; flag: an LDS int).  A wait
// that expires flags the launch's error word and answers no.
template <class A>
__device__ __forceinline__ bool leads_share_xcd(xw* words, int n, int i, int* flag, const A& a) {
  if (threadIdx.x == 0) {
    const unsigned x = __builtin_amdgcn_s_getreg((3 << 11) | 20) & 15u;   // XCC_ID, bits 3:0
    __hip_atomic_store(words + i, 0x100u | x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int same = 1;
    WaitBudget wb{wr_clock(), 0};
    for (int k = 0; k < n && same; ++k) {
      xw w;
      while (!((w = xpeek(words + k)) & 0x100u))
        if (!wait_ok(wb, a.err, a.limit, a.err)) {
          same = 0;
          break;
        }
      same = same && (w & 15u) == x;
    }
    *flag = same;
  }
  __syncthreads();
  return *flag != 0;
}
