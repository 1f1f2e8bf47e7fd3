// The masked dilated 1-D CNN that conditions the Subscale WaveRNN (Sec. 4.1,
// Sec. 5): for every utterance u, sub-tensor s and row (block of B samples)
// k, a Dx-wide conditioning vector computed from the previous sub-tensors'
// samples of rows k .. k + 124 (the mask keeps the future taps only).
//
// All rows of all sub-tensors are computed at once: every layer is one GEMM of
// M = utterances x B x rows activation rows against a weight matrix on the
// matrix cores (v_mfma_f32_16x16x32_bf16).  Weights are bf16; activations are
// fp32 in HBM and enter the matrix cores as a bf16 high part and a bf16
// remainder (two products per weight, about 16 significant bits), so the
// layers keep fp32-level accuracy.  A dilated convolution layer reads its
// three taps (rows k, k + d, k + 2d of the same sub-tensor, zero past the
// utterance's last row, as the mask of an utterance-long network has it)
// straight from the previous layer's rows, without an unfolded copy.  The
// network can also run over windows of rows (sampling runs it ahead in
// chunks): taps past a window are zero too, which changes only rows whose
// reach leaves the window.  Layer by layer:
//   input   r = Win x + bin         K = 2B (padded to 32)  N = Rc
//   conv l  a = relu(Wc [r_k | r_k+d | r_k+2d] + bc)  K = 3 Rc  N = Cc
//   proj l  r = r + (Wo a + bo)     K = Cc                 N = Rc
//   output  o = Wp r + bp           K = Rc                 N = Dx
#include "wr_kern.h"


namespace {

// Streamed runs: the sub-tensor and the utterance row of run row m (see CnnGemmArgs).
__device__ __forceinline__ int cnn_rng_row(const CnnGemmArgs& a, int m, int* s, int* blk) {
  const int b = m / a.rows;
  *s = a.out_s0 + b % a.B;
  *blk = (b / a.B) * a.out_B + *s;                  // (utterance, sub-tensor) of the whole-utterance arrays
  return a.lo[*s] + m % a.rows;
}

// A's piece of thread t for K-step kt: row t / 4 of the tile, inputs 8 (t % 4) .. +7 of the step.
__device__ __forceinline__ void cnn_load(const CnnGemmArgs& a, int m0, int n0, int kt, float4* x, uint4* wv) {
  const int t = threadIdx.x, row = t >> 2, oct = t & 3;
  const int m = m0 + row;
  const int kbase = kt * 32, tap = kbase / a.kin, col = kbase % a.kin + 8 * oct;
  bool ok;
  size_t sr;                                         // source row
  if (a.rng) {
    int s = 0, blk = 0;
    const int q = m < a.M ? cnn_rng_row(a, m, &s, &blk) + tap * a.dil : 0;   // the tap's utterance row
    ok = m < a.M && q < a.rows_utt;
    sr = a.src_abs ? (size_t)blk * a.rows_utt + q : (size_t)m;
  } else {
    const int kb = m % a.rows + tap * a.dil;         // row within the block of the tap
    const int64_t q = a.row0 + (int64_t)((m / a.rows) % a.B) * a.row_step + kb;   // its utterance row
    ok = m < a.M && kb < a.rows && q < a.rows_utt;
    sr = (size_t)(m + tap * a.dil);
  }
  if (ok) {
    const float4* p = (const float4*)(a.src + sr * a.kin + col);
    x[0] = p[0];
    x[1] = p[1];
  } else {
    x[0] = float4{0, 0, 0, 0};
    x[1] = float4{0, 0, 0, 0};
  }
  // W: column tile t / 64 of this workgroup's 8, lane t % 64
  *wv = a.w[((size_t)(n0 / 16 + (t >> 6)) * (a.K / 32) + kt) * 64 + (t & 63)];
}

__device__ __forceinline__ void cnn_stage(unsigned char* buf, const float4* x, uint4 wv) {
  const int t = threadIdx.x, row = t >> 2, oct = t & 3;
  const float v[8] = {x[0].x, x[0].y, x[0].z, x[0].w, x[1].x, x[1].y, x[1].z, x[1].w};
  bf16x8 hi, lo;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float h = __uint_as_float(__float_as_uint(v[e]) & 0xffff0000u);
    hi[e] = (__bf16)h;
    lo[e] = (__bf16)(v[e] - h);
  }
  // operand-A fragment of row tile row / 16: lane (row % 16) + 16 oct
  const int off = ((row >> 4) * 64 + (row & 15) + 16 * oct) * 16;
  *(bf16x8*)(buf + off) = hi;
  *(bf16x8*)(buf + 8 * WR_FRAG + off) = lo;
  *(uint4*)(buf + 16 * WR_FRAG + t * 16) = wv;
}

}  // namespace

// Workgroup b takes work item L = (b % 8) per_xcd + b / 8 (tile L mod tiles,
// group L / tiles when split): consecutive tiles (the column tiles of one row
// tile, which read the same activations) share an XCD and its L2.  Wave w
// computes rows 64 (w / 4) .. +63 and columns 32 (w % 4) .. +31 of the tile:
// 4 x 2 MFMA tiles, each as a high and a low product.  The K loop sums in
// groups of `group` K-steps, each group from zero, added in order: the same
// arithmetic whether one workgroup runs every group (a small GEMM has fewer
// tiles than CUs, and one tile's K loop would set its time) or each group
// runs on its own workgroup and wr_cnn_reduce adds them, so results never
// depend on how many rows a run has.
__device__ __forceinline__ void cnn_store(const CnnGemmArgs& a, int m0, int n0, const f32x4 (&v)[4][2], float* part) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wm = wave >> 2, wn = wave & 3;
  // lane l of tile (i, j) holds rows 4 (l / 16) .. +3, column l % 16
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = n0 + 32 * wn + 16 * j + (lane & 15);
    const float bn = part ? 0.0f : a.bias[n];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 64 * wm + 16 * i + 4 * (lane >> 4) + r;
        if (m >= a.M) continue;
        if (part) {
          part[(size_t)m * a.N + n] = v[i][j][r];
          continue;
        }
        size_t dm;
        if (a.rng) {
          int s, b2;
          const int q = cnn_rng_row(a, m, &s, &b2);
          if (q >= a.hi[s]) continue;                  // not a row of this run
          dm = a.dst_abs ? (size_t)b2 * a.rows_utt + q : (size_t)m;
        } else {
          const int blk = m / a.rows;
          dm = (size_t)((blk / a.B) * a.out_B + a.out_s0 + blk % a.B) * a.rows + m % a.rows;
        }
        float* d = a.dst + dm * a.N + n;
        const float x = v[i][j][r] + bn;
        *d = a.epi == 0 ? x : a.epi == 1 ? wr_relu(x) : *d + x;
      }
  }
}

__global__ __launch_bounds__(CNN_THREADS, 1) void wr_cnn_gemm(CnnGemmArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int b = blockIdx.x;
  const int L = (b % 8) * a.per_xcd + b / 8;
  if (b / 8 >= a.per_xcd || L >= a.tiles * a.split) return;
  const int tile = L % a.tiles, q = L / a.tiles;
  const int m0 = (tile % a.tiles_m) * CNN_TM, n0 = (tile / a.tiles_m) * CNN_TN;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, wm = wave >> 2, wn = wave & 3;
  f32x4 acc[4][2], grp[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = grp[i][j] = f32x4{0, 0, 0, 0};
  const int KT = a.K / 32;
  const int k_lo = a.split > 1 ? q * a.group : 0, k_hi = a.split > 1 ? min(KT, k_lo + a.group) : KT;
  float4 x[2];
  uint4 wv;
  cnn_load(a, m0, n0, k_lo, x, &wv);
  for (int kt = k_lo; kt < k_hi; ++kt) {
    unsigned char* buf = lds + (kt & 1) * CNN_LDS_BUF;
    cnn_stage(buf, x, wv);
    __syncthreads();
    if (kt + 1 < k_hi) cnn_load(a, m0, n0, kt + 1, x, &wv);   // in flight during the products
    bf16x8 bw[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) bw[j] = *(const bf16x8*)(buf + (16 + 2 * wn + j) * WR_FRAG + lane * 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bf16x8 ah = *(const bf16x8*)(buf + (4 * wm + i) * WR_FRAG + lane * 16);
      const bf16x8 al = *(const bf16x8*)(buf + (8 + 4 * wm + i) * WR_FRAG + lane * 16);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        grp[i][j] = mfma(ah, bw[j], grp[i][j]);
        grp[i][j] = mfma(al, bw[j], grp[i][j]);
      }
    }
    if ((kt + 1) % a.group == 0 || kt + 1 == KT) {   // a group ends: acc = acc + g (the first: acc = g)
      const bool first = kt + 1 <= a.group;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = first ? grp[i][j] : acc[i][j] + grp[i][j];
          grp[i][j] = f32x4{0, 0, 0, 0};
        }
    }
  }
  cnn_store(a, m0, n0, acc, a.split > 1 ? a.part + (size_t)q * a.M * a.N : nullptr);
}

// Split GEMMs: out = ((part[0] + part[1]) + part[2]) + ... + bias, then the
// epilogue, as wr_cnn_gemm's own when one workgroup runs every group.
__global__ void wr_cnn_reduce(CnnGemmArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)a.M * a.N) return;
  const int m = (int)(idx / a.N), n = (int)(idx % a.N);
  float v = a.part[idx];
  for (int q = 1; q < a.split; ++q) v = v + a.part[(size_t)q * a.M * a.N + idx];
  size_t dm;
  if (a.rng) {
    int s, b2;
    const int q = cnn_rng_row(a, m, &s, &b2);
    if (q >= a.hi[s]) return;                        // not a row of this run
    dm = a.dst_abs ? (size_t)b2 * a.rows_utt + q : (size_t)m;
  } else {
    const int blk = m / a.rows;
    dm = (size_t)((blk / a.B) * a.out_B + a.out_s0 + blk % a.B) * a.rows + m % a.rows;
  }
  float* d = a.dst + dm * a.N + n;
  const float x = v + a.bias[n];
  *d = a.epi == 0 ? x : a.epi == 1 ? wr_relu(x) : *d + x;
}

// Input rows of a window of `win` rows per (utterance u, sub-tensor s) for the
// sub-tensors s0 .. s0 + nsb - 1: row m = (u nsb + s - s0) win + k is
// utterance row q = row0 + s row_step + k.  x[m][2z],
// x[m][2z + 1] = the scaled (c, f) of sample B q + z for z < s (the previous
// sub-tensors of row q) when q is a row of the utterance and sub-tensor z has
// made it (q <= front0 + z front_step); zero otherwise and in the padding up
// to kin.
__global__ void wr_cnn_input(CnnInputArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)a.M * a.kin) return;
  const int m = (int)(idx / a.kin), ch = (int)(idx % a.kin);
  const int k = m % a.win, s = a.s0 + (m / a.win) % a.nsb, u = m / a.win / a.nsb, z = ch >> 1;
  const int64_t q = a.rng ? (int64_t)a.lo[s] + k : a.row0 + (int64_t)s * a.row_step + k;
  float v = 0.0f;
  if (z < s && q >= 0 && q < a.rows && q <= a.front0 + (int64_t)z * a.front_step) {
    const int smp = a.seq[(size_t)u * a.n_samples + (size_t)a.B * q + z];
    v = wr_scale((ch & 1) ? (smp & 255) : (smp >> 8));
  }
  a.x[idx] = v;
}

const void* wr_cnn_gemm_ptr() { return (const void*)wr_cnn_gemm; }
const void* wr_cnn_input_ptr() { return (const void*)wr_cnn_input; }
const void* wr_cnn_reduce_ptr() { return (const void*)wr_cnn_reduce; }
