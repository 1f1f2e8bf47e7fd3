// Single-workgroup WaveRNN sampler for small hidden sizes (all weights fit in
// one CU's LDS as fp32).  One workgroup per utterance.  It evaluates Eq. 2 and
// the dual softmax in one fixed order -- every dot product is an fma chain in
// increasing index order from +0, running sums of the softmax weights are
// sequential -- so its samples are deterministic and reproducible bit for bit
// by any implementation of the same order.
#include "wr_device.h"
#include "wr_layout.h"
#include "wr_args.h"

// fma chain over n terms: w[j * ws] * x[j], j increasing, from +0.
__device__ __forceinline__ float chain(const float* w, int ws, const float* x, int n) {
  float acc = 0.0f;
  for (int j = 0; j < n; ++j) acc = __builtin_fmaf(w[j * ws], x[j], acc);
  return acc;
}

// Gates of units [lo, hi) (Eq. 2, masked I*): one thread per unit.
__device__ __forceinline__ void small_units(const SmallLayout& L, float* s, int lo, int hi, float x0, float x1,
                                            float x2, bool fine) {
  const int H = L.H;
  for (int i = lo + (int)threadIdx.x; i < hi; i += blockDim.x) {
    float ix[3];
#pragma unroll
    for (int g = 0; g < 3; ++g) {
      const float* I = s + L.I + (g * H + i) * 3;
      float acc = 0.0f;
      acc = __builtin_fmaf(I[0], x0, acc);
      acc = __builtin_fmaf(I[1], x1, acc);
      if (fine) acc = __builtin_fmaf(I[2], x2, acc);
      ix[g] = acc;
    }
    const float* G = s + L.G;
    const float* add = s + L.add;
    float au = G[0 * H + i] + (ix[0] + add[0 * H + i]);
    float ar = G[1 * H + i] + (ix[1] + add[1 * H + i]);
    float u = wr_sigmoid(au);
    float r = wr_sigmoid(ar);
    float e = wr_tanh(__builtin_fmaf(r, G[2 * H + i], ix[2] + add[2 * H + i]));
    s[L.hn + i] = __builtin_fmaf(u, s[L.h + i], (1.0f - u) * e);
  }
}

// One output head (Eq. 2): z = Ob relu(Oa y + ba) + bb.  Oa, Ob stored transposed.
__device__ __forceinline__ void small_head(const SmallLayout& L, float* s, int Oat, int ba, int Obt, int bb,
                                           const float* y) {
  const int Hh = L.H / 2;
  for (int k = threadIdx.x; k < Hh; k += blockDim.x) s[L.hid + k] = wr_relu(chain(s + Oat + k, Hh, y, Hh) + s[ba + k]);
  __syncthreads();
  for (int v = threadIdx.x; v < WR_CLASSES; v += blockDim.x)
    s[L.z + v] = chain(s + Obt + v, WR_CLASSES, s + L.hid, Hh) + s[bb + v];
  __syncthreads();
}

// Inverse-CDF draw from softmax(z) with uniform u (z in LDS, 256 threads).
// Returns the class in every thread; *lse = max z + log(sum exp(z - max z)).
__device__ int small_draw(const SmallLayout& L, float* s, float u, int forced, float* lse) {
  __shared__ float red[8];
  __shared__ int cnt[8];
  const int v = threadIdx.x, wave = v >> 6, lane = v & 63;
  float zv = s[L.z + v];
  float m = wave_max(zv);
  if (lane == 0) red[wave] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float wv = wr_exp(zv - m);
  s[L.w + v] = wv;
  __syncthreads();
  if (v == 0) {
    float run = 0.0f;
    for (int k = 0; k < WR_CLASSES; ++k) {
      run = run + s[L.w + k];
      s[L.C + k] = run;
    }
  }
  __syncthreads();
  const float Z = s[L.C + WR_CLASSES - 1];
  *lse = m + logf(Z);
  if (forced >= 0) return forced;
  const float thr = u * Z;
  int below = s[L.C + v] <= thr;
  int nb = __popcll(__ballot(below));
  int last = wv > 0.0f ? v : -1;
  last = wave_max_i(last);
  if (lane == 0) {
    cnt[wave] = nb;
    cnt[4 + wave] = last;
  }
  __syncthreads();
  int count = cnt[0] + cnt[1] + cnt[2] + cnt[3];
  if (count == WR_CLASSES) count = max(max(cnt[4], cnt[5]), max(cnt[6], cnt[7]));
  __syncthreads();
  return count;
}

extern "C" __global__ __launch_bounds__(256, 1) void wr_small_kernel(SmallArgs a) {
  extern __shared__ __align__(16) float s[];
  const SmallLayout L = small_layout(a.H);
  const int H = a.H, Hh = H / 2, tid = threadIdx.x;
  const int st = blockIdx.x;  // utterance = Philox stream
  {  // weights -> LDS
    const uint4* src = (const uint4*)a.image;
    uint4* dst = (uint4*)s;
    for (int i = tid; i < L.image_floats / 4; i += blockDim.x) dst[i] = src[i];
  }
  for (int i = tid; i < H; i += blockDim.x) s[L.h + i] = a.h_in ? a.h_in[(size_t)st * H + i] : 0.0f;
  __shared__ int cprev, fprev;
  if (tid == 0) {
    cprev = a.c_in ? a.c_in[st] : 128;
    fprev = a.f_in ? a.f_in[st] : 0;
  }
  __syncthreads();
  int64_t cur_frame = -1;
  for (int64_t t = 0; t < a.T; ++t) {
    const int64_t n = a.t0 + t;
    // gate additive term: bias (+ conditioning of the frame)
    int64_t fr = a.Dc > 0 ? n / a.frame_len : 0;
    if (fr >= a.n_frames && a.Dc > 0) fr = a.n_frames - 1;
    if (fr != cur_frame) {
      cur_frame = fr;
      for (int row = tid; row < 3 * H; row += blockDim.x) {
        float b = s[L.bias + row];
        float v = b;
        if (a.Dc > 0) v = chain(a.Wc + (size_t)row * a.Dc, 1, a.feat + ((size_t)st * a.n_frames + fr) * a.Dc, a.Dc) + b;
        s[L.add + row] = v;
      }
    }
    // G = R h (R stored transposed: column-major rows)
    for (int row = tid; row < 3 * H; row += blockDim.x) s[L.G + row] = chain(s + L.Rt + row, 3 * H, s + L.h, H);
    __syncthreads();
    const float x0 = wr_scale(cprev), x1 = wr_scale(fprev);
    const int64_t o = (int64_t)st * a.T + t;
    const int tc = a.target ? (a.target[o] >> 8) : -1;
    const int tf = a.target ? (a.target[o] & 255) : -1;
    // coarse half, coarse head, coarse draw
    small_units(L, s, 0, Hh, x0, x1, 0.0f, false);
    __syncthreads();
    small_head(L, s, L.O1t, L.b1, L.O2t, L.b2, s + L.hn);
    if (a.zc_out) a.zc_out[o * WR_CLASSES + tid] = s[L.z + tid];
    float uc, uf;
    wr_uniforms(a.seed, (uint64_t)st, (uint64_t)n, &uc, &uf);
    float lse_c, lse_f;
    const int c = small_draw(L, s, uc, tc, &lse_c);
    const float zc_c = s[L.z + c];
    // fine half sees c_t, fine head, fine draw
    small_units(L, s, Hh, H, x0, x1, wr_scale(c), true);
    __syncthreads();
    small_head(L, s, L.O3t, L.b3, L.O4t, L.b4, s + L.hn + Hh);
    if (a.zf_out) a.zf_out[o * WR_CLASSES + tid] = s[L.z + tid];
    const int f = small_draw(L, s, uf, tf, &lse_f);
    if (tid == 0) {
      if (a.out) a.out[o] = (uint16_t)(256 * c + f);
      if (a.nll_out) a.nll_out[o] = (lse_c - zc_c) + (lse_f - s[L.z + f]);
      cprev = c;
      fprev = f;
    }
    for (int i = tid; i < H; i += blockDim.x) s[L.h + i] = s[L.hn + i];
    __syncthreads();
  }
  if (a.h_out)
    for (int i = tid; i < H; i += blockDim.x) a.h_out[(size_t)st * H + i] = s[L.h + i];
  if (tid == 0) {
    if (a.c_out) a.c_out[st] = (uint8_t)cprev;
    if (a.f_out) a.f_out[st] = (uint8_t)fprev;
  }
}

const void* wr_small_kernel_ptr() { return (const void*)wr_small_kernel; }

// Uniforms exactly as the sampling kernels draw them (for tests).
extern "C" __global__ void wr_uniforms_kernel(uint64_t seed, uint64_t stream, int64_t t0, int64_t n, float* out) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float uc, uf;
  wr_uniforms(seed, stream, (uint64_t)(t0 + i), &uc, &uf);
  out[2 * i] = uc;
  out[2 * i + 1] = uf;
}

const void* wr_uniforms_kernel_ptr() { return (const void*)wr_uniforms_kernel; }
