// Device helpers of libwavernn (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef unsigned long long u64;

#define WR_CLASSES 256

// ---------------------------------------------------------------------------
// Elementary functions.  exp(y): Cody-Waite reduction y = k ln2 + r with ln 2
// split into a 15-significant-bit head and a tail (Cody & Waite, 1980), then
// the degree-7 Taylor polynomial of e^r in Horner form with fma, scaled by an
// exactly built 2^k.  The same evaluation order is used on every path so the
// fp32 single-workgroup kernel is deterministic.
//   LN2_HI = 22713 * 2^-15        (ln 2 truncated to 15 significant bits)
//   LN2_LO = fp32(ln 2 - LN2_HI)  LOG2E = fp32(1 / ln 2)   C_i = fp32(1 / i!)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wr_exp(float y) {
  const float LOG2E = 0x1.715476p+0f;
  const float LN2_HI = 0x1.62e4p-1f;
  const float LN2_LO = 0x1.7f7d1cp-20f;
  if (y != y) return y;
  if (y < -86.0f) return 0.0f;   // below 2^-124: flushed so no result is subnormal
  if (y > 88.0f) return __builtin_inff();
  float k = __builtin_rintf(y * LOG2E);
  float r = __builtin_fmaf(-k, LN2_HI, y);
  r = __builtin_fmaf(-k, LN2_LO, r);
  float p = 0x1.a01a02p-13f;                // 1/7!
  p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);  // 1/6!
  p = __builtin_fmaf(p, r, 0x1.111112p-7f);   // 1/5!
  p = __builtin_fmaf(p, r, 0x1.555556p-5f);   // 1/4!
  p = __builtin_fmaf(p, r, 0x1.555556p-3f);   // 1/3!
  p = __builtin_fmaf(p, r, 0.5f);             // 1/2!
  p = __builtin_fmaf(p, r, 1.0f);             // 1/1!
  p = __builtin_fmaf(p, r, 1.0f);             // 1/0!
  int ki = (int)k;
  float two_k = __uint_as_float((uint32_t)(ki + 127) << 23);
  return p * two_k;
}

// Standard sigmoid and tanh of Eq. 2 written through wr_exp.
__device__ __forceinline__ float wr_sigmoid(float x) { return 1.0f / (1.0f + wr_exp(-x)); }

__device__ __forceinline__ float wr_tanh(float x) {
  float a = __builtin_fabsf(x);
  float q = wr_exp(-2.0f * a);
  float t = (1.0f - q) / (1.0f + q);
  return __builtin_copysignf(t, x);
}

__device__ __forceinline__ float wr_relu(float v) { return v > 0.0f ? v : 0.0f; }

// A byte in [0, 255] scaled to [-1, 1] (Sec. 2): (2v - 255) / 255, correctly rounded.
__device__ __forceinline__ float wr_scale(int v) { return (float)(2 * v - 255) / 255.0f; }

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw: "Parallel random numbers: as easy
// as 1, 2, 3", SC'11): 10 rounds of two 64x64->128 multiplies, key bumped by
// the Weyl constants between rounds.
// ---------------------------------------------------------------------------
__host__ __device__ __forceinline__ void wr_mulhilo(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
#if defined(__HIP_DEVICE_COMPILE__)
  *hi = __umul64hi(a, b);
  *lo = a * b;
#else
  unsigned __int128 p = (unsigned __int128)a * b;
  *hi = (uint64_t)(p >> 64);
  *lo = (uint64_t)p;
#endif
}

__host__ __device__ __forceinline__ void wr_philox(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0,
                                                   uint64_t k1, uint64_t out[4]) {
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += 0x9E3779B97F4A7C15ULL;
      k1 += 0xBB67AE8584CAA73BULL;
    }
    uint64_t hi0, lo0, hi1, lo1;
    wr_mulhilo(0xD2E7470EE14C6C93ULL, c0, &hi0, &lo0);
    wr_mulhilo(0xCA5A826395121157ULL, c2, &hi1, &lo1);
    uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

// Coarse and fine uniforms of absolute step t on a stream: words 0 and 1 of the
// block at counter (t, stream, 0, 0), key (seed, 0); 24 top bits -> [0, 1).
__host__ __device__ __forceinline__ void wr_uniforms(uint64_t seed, uint64_t stream, uint64_t t, float* uc, float* uf) {
  uint64_t w[4];
  wr_philox(t, stream, 0, 0, seed, 0, w);
  *uc = (float)(uint32_t)(w[0] >> 40) * (1.0f / 16777216.0f);
  *uf = (float)(uint32_t)(w[1] >> 40) * (1.0f / 16777216.0f);
}

// ---------------------------------------------------------------------------
// bf16 weights: a 32-bit word holds two bf16 (element 2j in the low half).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// ---------------------------------------------------------------------------
// Inter-workgroup exchange.  A 32-bit word carries an fp32 value whose lowest
// mantissa bit is replaced by the parity of the tag (step number) that
// produced it.  Every consumer reads every word it uses once per step, and the
// dependency chain keeps a producer at most one step ahead of any consumer of
// its words, so a word is either the previous step's (other parity) or the
// awaited one: one bit tells them apart, and each exchange moves half the
// bytes of a value + full-tag pair.  Aligned 32-bit atomic accesses are
// single-copy atomic; agent-scope relaxed accesses keep the words coherent
// across all XCDs (each XCD has its own L2).  The cost is 1 ulp on the value.
// ---------------------------------------------------------------------------
typedef uint32_t xw;
__device__ __forceinline__ void xpub(xw* p, uint32_t tag, float v) {
  const xw w = (__float_as_uint(v) & ~1u) | (tag & 1u);
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ xw xpeek(const xw* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool xok(xw w, uint32_t tag) { return ((w ^ tag) & 1u) == 0; }
__device__ __forceinline__ float xval(xw w) { return __uint_as_float(w & ~1u); }
// A word that only workgroups on the writer's own XCD read (`local`, see
// leads_share_xcd) is published with a plain store: it stays in that XCD's L2,
// where the readers' coherent loads find it, a shorter hop than a store
// written through to memory.  Otherwise as xpub.
__device__ __forceinline__ void xpub_l(xw* p, uint32_t tag, float v, bool local) {
  const xw w = (__float_as_uint(v) & ~1u) | (tag & 1u);
  if (local) __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  else __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Two adjacent words (p 8-byte aligned) written and read as one 64-bit access.
__device__ __forceinline__ void xpub2(xw* p, uint32_t tag, float v0, float v1) {
  const uint64_t w = (uint64_t)((__float_as_uint(v0) & ~1u) | (tag & 1u)) |
                     (uint64_t)((__float_as_uint(v1) & ~1u) | (tag & 1u)) << 32;
  __hip_atomic_store((uint64_t*)p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t xpeek2(const xw* p) {
  return __hip_atomic_load((const uint64_t*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool xok2(uint64_t w, uint32_t tag) { return xok((xw)w, tag) && xok((xw)(w >> 32), tag); }

// Four adjacent words (16-byte aligned) read by one 16-byte buffer load with
// the coherence bit of the agent-scope loads above (sc1).  Each 32-bit word
// of it is read whole, but the four need not be from one moment, so each
// keeps its own tag.  The resource bounds every access to `bytes` from base
// (reads beyond return zero).  The compiler takes such a load for a pure
// function of its operands, so a polling loop must build the resource in
// every round from a base it cannot see through (xopaque), or the loads are
// hoisted out of the loop.
typedef uint32_t xw4 __attribute__((ext_vector_type(4)));
template <class T>
__device__ __forceinline__ T* xopaque(T* p) {
  asm volatile("" : "+s"(p));
  return p;
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t xrsrc(const xw* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, 0, (int)bytes, 0x00020000);   // raw 32-bit data (gfx9)
}
__device__ __forceinline__ xw4 xpeek4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 16);   // cache policy 16: sc1
}
__device__ __forceinline__ bool xok4(xw4 w, uint32_t tag) {
  return (((w.x ^ tag) | (w.y ^ tag) | (w.z ^ tag) | (w.w ^ tag)) & 1u) == 0;
}

// A value as a reader of the exchange sees it (so that state handed in by the
// caller enters a computation exactly as the exchanged values do).
__device__ __forceinline__ float xround(float v) { return __uint_as_float(__float_as_uint(v) & ~1u); }

__device__ __forceinline__ u64 wr_clock() { return __builtin_amdgcn_s_memrealtime(); }  // 100 MHz

// Error word bits set by kernels.
#define WR_ERR_TIMEOUT 1u
#define WR_ERR_TAG 2u
#define WR_ERR_PLACEMENT 4u

// Bounded wait bookkeeping: every wait gives up after `limit` ticks of the
// 100 MHz clock, or when another workgroup has already flagged an error.
struct WaitBudget {
  u64 start;
  unsigned spins;
};
__device__ __forceinline__ bool wait_ok(WaitBudget& wb, const unsigned* err, u64 limit, unsigned* err_w) {
  ++wb.spins;
  if ((wb.spins & 63u) == 0) {
    if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return false;
    if (wr_clock() - wb.start > limit) {
      atomicOr(err_w, WR_ERR_TIMEOUT);
      return false;
    }
  }
  return true;
}

// ---------------------------------------------------------------------------
// Wave64 reductions (xor butterflies through ds_swizzle / DPP via shfl).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ int wave_max_i(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = max(v, __shfl_xor(v, m, 64));
  return v;
}
