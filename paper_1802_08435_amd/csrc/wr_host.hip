// Host side of libwavernn: validation, weight packing, launch plans, C ABI.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "wavernn.h"
#include "wr_args.h"
#include "wr_layout.h"

namespace {

thread_local std::string g_err;

wavernn_status fail(wavernn_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
wavernn_status fail(wavernn_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIPOK(call)                                                                        \
  do {                                                                                     \
    hipError_t e_ = (call);                                                                \
    if (e_ != hipSuccess) return fail(WAVERNN_E_HIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

// fp32 -> bf16, round to nearest even (NaN stays NaN).
uint16_t f2bf(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
float bf2f(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

enum Path { PATH_SMALL = 0, PATH_PERSIST = 1, PATH_BATCHED = 2 };
constexpr int PATH_SPARSE_ID = 3, PATH_CONCURRENT_ID = 4, PATH_FUSED_ID = 5;   // wavernn_model_path's ids of the variants
#define WR_FAN 4   // concurrent batch-1 launches: the caller's stream and 3 internal ones (HIP's default
                   // of 4 hardware queues gives each its own)

const u64 kWaitTicks = 200000000ull;  // 2 s of the 100 MHz clock per wait

}  // namespace

struct wavernn_model {
  wavernn_config cfg;
  int device = 0;
  Path path = PATH_SMALL;
  std::vector<void*> allocs;
  unsigned* d_err = nullptr;
  // small path
  float* d_image = nullptr;
  float* d_Wc = nullptr;
  SmallLayout sl;
  // persistent path
  PersistPlan plan;
  const void* pk = nullptr;          // kernel instantiation for the plan
  bool sparse = false;               // block-sparse units
  bool fused = false;                // Fused Subscale WaveRNN 2x heads (Sec. 4.4)
  uint4 *d_hw = nullptr, *d_uw = nullptr, *d_ur = nullptr;
  uint4* d_mw = nullptr;             // mirror fragments (dense batch-1 plan)
  float *d_I = nullptr, *d_bias = nullptr, *d_b1 = nullptr, *d_b2 = nullptr, *d_b3 = nullptr, *d_b4 = nullptr;
  float* d_cb = nullptr;             // [cb_cap][3H] bias + conditioning per frame
  int64_t cb_cap = 0;
  xw* d_xc = nullptr;                // exchange words (zeroed as 64-bit pairs)
  int solo_hx = 0, solo_uxm = 255;   // placement of launches that run one at a time (wavernn_tune)
  // teacher-forced scoring on the dense batch-1 plan: the recurrence kernel, the
  // output layers as GEMM fragments (O1 [NP][Hh], O2 [256][NP], O3, O4; NP = Hh
  // rounded up to 128) and biases, and the buffers of a call
  const void* sk = nullptr;
  const void* smk = nullptr;         // the scoring recurrence for up to 8 utterances at once (null: none)
  xw* d_sxc[WR_FAN] = {};            // its exchange words [2][8][H] per slot
  float* d_scb[WR_FAN] = {};         // its tables [8][frames][3H] per slot
  int64_t scb_cap = 0;               // floats of each
  uint4* d_srw = nullptr;             // [H/16][3][H/32][64] R fragments of the scoring recurrence
  uint4* d_sw = nullptr;
  float* d_sb = nullptr;
  size_t sw_off[4] = {}, sb_off[4] = {};
  int sc_np = 0;
  float* d_traj = nullptr;            // [2][rows][Hh] h after each step (coarse half, then fine half)
  int64_t traj_cap = 0;               // rows
  float *d_so = nullptr, *d_sz = nullptr;   // [rows][NP] first-layer output, [2][rows][256] logits
  int64_t so_cap = 0;                       // rows of d_so and d_sz (at most one chunk of the output layers)
  u64* trace = nullptr;
  int64_t trace_steps = 0;
  // concurrent batch-1 launches: a few utterances, each on its own persistent
  // grid and its own internal stream, all grids co-resident at once
  int nfan = 0;                      // most utterances served this way (0: none)
  bool score_fan = false;            // scoring runs up to nfan utterances' recurrence grids side by side
  hipStream_t fan_st[WR_FAN - 1] = {};  // launches 1 .. (launch 0 runs on the caller's stream)
  hipEvent_t fan_fork = nullptr, fan_join[WR_FAN - 1] = {};
  xw* d_fxc[WR_FAN] = {};            // exchange words of launch i
  float* d_fcb[WR_FAN] = {};         // [fcb_cap][3H] bias + conditioning of launch i
  int64_t fcb_cap = 0;
  // conditioning CNN of a subscale model (Sec. 4.1): weight fragments of the
  // input layer, then per layer the convolution and the projection, then the
  // output layer, in one buffer; biases likewise; activations grown on demand
  struct Cnn {
    int Rc = 0, Cc = 0, layers = 0, kin = 32;
    uint4* w = nullptr;
    float* bias = nullptr;
    std::vector<size_t> woff, boff;   // [input, conv 0, proj 0, conv 1, ..., output] in uint4 / floats
    float *x = nullptr, *r = nullptr, *act = nullptr;
    int64_t cap = 0;                   // activation rows the buffers hold
    float* part = nullptr;             // per-group partial products of split GEMMs
    int64_t part_cap = 0;              // floats
    float* rfull = nullptr;            // streamed sampling: residual activations [U][B][rows][Rc]
    int64_t rfull_cap = 0;             // floats
  } cnn;
  bool has_cnn = false;
  int64_t cnn_chunk = 0, cnn_win = 0;   // sampling: steps per chunk, CNN window rows
  float* d_ctab = nullptr;              // context table [max_streams][B][rows or window][Dx]
  int64_t ctab_cap = 0;                 // floats
  wavernn_state cnn_state[2] = {};      // state between chunks (ping-pong)
  // batched path (several utterances per launch)
  bool has_batch = false;
  BatchPlan bplan;
  uint4 *d_buw = nullptr, *d_bur = nullptr, *d_bux = nullptr;
  xw* d_bxc = nullptr;
  float* d_bcb = nullptr;            // [streams][frames][3H]
  size_t bcb_cap = 0;                // floats

  template <typename T>
  wavernn_status alloc(T** p, size_t bytes) {
    void* q = nullptr;
    if (hipMalloc(&q, bytes ? bytes : 16) != hipSuccess) {
      (void)hipGetLastError();
      return fail(WAVERNN_E_OOM, "device allocation of %zu bytes failed", bytes);
    }
    allocs.push_back(q);
    *p = (T*)q;
    return WAVERNN_OK;
  }
  template <typename T>
  wavernn_status upload(T** p, const void* host, size_t bytes) {
    wavernn_status s = alloc(p, bytes);
    if (s != WAVERNN_OK) return s;
    HIPOK(hipMemcpy(*p, host, bytes, hipMemcpyHostToDevice));
    return WAVERNN_OK;
  }
  ~wavernn_model() {
    for (int i = 0; i < WR_FAN - 1; ++i) {
      if (fan_st[i]) (void)hipStreamSynchronize(fan_st[i]);
      if (fan_st[i]) (void)hipStreamDestroy(fan_st[i]);
      if (fan_join[i]) (void)hipEventDestroy(fan_join[i]);
    }
    if (fan_fork) (void)hipEventDestroy(fan_fork);
    for (void* q : allocs) (void)hipFree(q);
  }
};

namespace {

// Weight value as the model stores it (bf16-rounded in BF16 mode).
struct Rounder {
  bool bf16;
  float operator()(float v) const { return bf16 ? bf2f(f2bf(v)) : v; }
};

// Future horizon of a subscale model (Sec. 4.2), -1 for lockstep rows or B = 1.
static int horizon_of(const wavernn_config& c) { return c.subscale > 1 ? c.future_horizon : -1; }
// Steps by which the units form a horizon context ahead of its use (0 without a horizon).
static int lead_of(const wavernn_config& c) { return horizon_of(c) >= 0 ? c.context_lead : 0; }

wavernn_status validate_config(const wavernn_config* c, const wavernn_weights* w) {
  if (!c || !w) return fail(WAVERNN_E_INVALID, "null config or weights");
  if (c->hidden <= 0 || (c->hidden & 1)) return fail(WAVERNN_E_INVALID, "hidden must be positive and even (got %d)", c->hidden);
  if (c->hidden > 4096) return fail(WAVERNN_E_INVALID, "hidden %d above 4096", c->hidden);
  if (c->cond_dim < 0 || c->cond_dim > 1024) return fail(WAVERNN_E_INVALID, "cond_dim %d out of range", c->cond_dim);
  if (c->cond_dim > 0 && c->frame_len <= 0) return fail(WAVERNN_E_INVALID, "frame_len must be > 0 with conditioning");
  if (c->subscale < 1 || c->subscale > 64) return fail(WAVERNN_E_INVALID, "subscale %d out of range", c->subscale);
  if (c->subscale == 1 && c->ctx_dim != 0) return fail(WAVERNN_E_INVALID, "ctx_dim must be 0 when subscale is 1");
  if (c->subscale > 1 && !c->fused && (c->ctx_dim <= 0 || (c->ctx_dim & 1) || c->ctx_dim > 1024))
    return fail(WAVERNN_E_INVALID, "ctx_dim must be even and in (0, 1024] with subscale");
  if (c->subscale > 1 && (c->future_horizon < -1 || c->future_horizon > 1024))
    return fail(WAVERNN_E_INVALID, "future_horizon %d out of [-1, 1024]", c->future_horizon);
  if (c->subscale > 1 && c->future_horizon >= 0 && c->ctx_dim % 4)
    return fail(WAVERNN_E_INVALID, "ctx_dim must be a multiple of 4 with a future horizon");
  if (c->subscale > 1 && (c->context_lead < 0 || c->context_lead > 3 || (c->future_horizon < 0 && c->context_lead)))
    return fail(WAVERNN_E_INVALID, "context_lead %d: must be in [0, 3], and 0 without a future horizon",
                c->context_lead);
  if (c->subscale > 1 && c->context_lead > 0)
    return fail(WAVERNN_E_UNSUPPORTED, "context_lead %d: switched off (a traced launch had a bounded wait expire "
                "with a lead of 1 and the cause is not found; the lead-0 schedule is unaffected)", c->context_lead);
  if (c->weight_dtype != WAVERNN_F32 && c->weight_dtype != WAVERNN_BF16) return fail(WAVERNN_E_INVALID, "bad weight_dtype");
  if (c->r_format < WAVERNN_R_DENSE || c->r_format > WAVERNN_R_BSR_16X1) return fail(WAVERNN_E_INVALID, "bad r_format");
  if (c->max_streams < 1 || c->max_streams > 64) return fail(WAVERNN_E_INVALID, "max_streams must be in [1, 64]");
  if (c->fused != 0 && c->fused != 1) return fail(WAVERNN_E_INVALID, "fused must be 0 or 1");
  if (c->fused && (c->subscale != 2 || c->ctx_dim != 0 || c->future_horizon < 0 || c->context_lead != 0 ||
                   c->r_format != WAVERNN_R_DENSE || c->hidden % 4))
    return fail(WAVERNN_E_INVALID, "fused 2x: needs subscale 2, ctx_dim 0, future_horizon >= 0, context_lead 0, "
                "dense R and hidden a multiple of 4");
  if (!w->R || !w->I || !w->b || !w->O1 || !w->b1 || !w->O2 || !w->b2 ||
      (!c->fused && (!w->O3 || !w->b3 || !w->O4 || !w->b4)))
    return fail(WAVERNN_E_INVALID, "a required weight array is null");
  if (c->cond_dim > 0 && !w->W_cond) return fail(WAVERNN_E_INVALID, "W_cond is null with cond_dim > 0");
  if (w->ctx_cnn) {
    const wavernn_ctx_cnn* n = w->ctx_cnn;
    if (c->subscale < 2 || c->fused || c->future_horizon < 0)
      return fail(WAVERNN_E_INVALID, "ctx_cnn: needs a subscale model with a future horizon");
    if (n->res_channels <= 0 || n->res_channels % 128 || n->conv_channels <= 0 || n->conv_channels % 128 ||
        n->layers < 0 || n->layers > 64 || c->ctx_dim % 128 || 2 * c->subscale > 1024)
      return fail(WAVERNN_E_INVALID, "ctx_cnn: res/conv channels and ctx_dim must be positive multiples of 128, "
                  "layers in [0, 64]");
    if (!n->Win || !n->bin || !n->Wp || !n->bp || (n->layers > 0 && (!n->Wc || !n->bc || !n->Wo || !n->bo)))
      return fail(WAVERNN_E_INVALID, "ctx_cnn: a weight array is null");
  }
  if (c->ctx_dim > 0 && !w->W_ctx) return fail(WAVERNN_E_INVALID, "W_ctx is null with ctx_dim > 0");
  if (c->r_format != WAVERNN_R_DENSE) {
    int bh = c->r_format == WAVERNN_R_BSR_4X4 ? 4 : 16, bw = c->r_format == WAVERNN_R_BSR_4X4 ? 4 : 1;
    if (c->hidden % bh || c->hidden % bw) return fail(WAVERNN_E_INVALID, "hidden not a multiple of the block shape");
    if (!w->R_block_mask) return fail(WAVERNN_E_INVALID, "R_block_mask is null for a block-sparse format");
  }
  return WAVERNN_OK;
}

// Effective dense R entry (pruned blocks read as zero).
struct REff {
  const wavernn_config* c;
  const wavernn_weights* w;
  float operator()(int row, int col) const {
    const int H = c->hidden;
    if (c->r_format != WAVERNN_R_DENSE) {
      int bh = c->r_format == WAVERNN_R_BSR_4X4 ? 4 : 16, bw = c->r_format == WAVERNN_R_BSR_4X4 ? 4 : 1;
      int g = row / H, i = row % H;
      size_t mi = ((size_t)g * (H / bh) + i / bh) * (H / bw) + col / bw;
      if (!w->R_block_mask[mi]) return 0.0f;
    }
    return w->R[(size_t)row * H + col];
  }
};

wavernn_status build_small(wavernn_model* m, const wavernn_weights* w) {
  const wavernn_config& c = m->cfg;
  const int H = c.hidden, Hh = H / 2;
  const SmallLayout L = small_layout(H);
  m->sl = L;
  Rounder rd{c.weight_dtype == WAVERNN_BF16};
  REff R{&m->cfg, w};
  std::vector<float> img(L.image_floats, 0.0f);
  for (int row = 0; row < 3 * H; ++row)
    for (int j = 0; j < H; ++j) img[L.Rt + (size_t)j * 3 * H + row] = rd(R(row, j));
  for (int row = 0; row < 3 * H; ++row) {
    int i = row % H;
    for (int q = 0; q < 3; ++q) img[L.I + row * 3 + q] = (q == 2 && i < Hh) ? 0.0f : rd(w->I[row * 3 + q]);
    img[L.bias + row] = rd(w->b[row]);
  }
  for (int k = 0; k < Hh; ++k)
    for (int j = 0; j < Hh; ++j) {
      img[L.O1t + j * Hh + k] = rd(w->O1[(size_t)k * Hh + j]);
      img[L.O3t + j * Hh + k] = rd(w->O3[(size_t)k * Hh + j]);
    }
  for (int v = 0; v < 256; ++v)
    for (int j = 0; j < Hh; ++j) {
      img[L.O2t + j * 256 + v] = rd(w->O2[(size_t)v * Hh + j]);
      img[L.O4t + j * 256 + v] = rd(w->O4[(size_t)v * Hh + j]);
    }
  for (int k = 0; k < Hh; ++k) {
    img[L.b1 + k] = rd(w->b1[k]);
    img[L.b3 + k] = rd(w->b3[k]);
  }
  for (int v = 0; v < 256; ++v) {
    img[L.b2 + v] = rd(w->b2[v]);
    img[L.b4 + v] = rd(w->b4[v]);
  }
  wavernn_status s = m->upload(&m->d_image, img.data(), img.size() * 4);
  if (s != WAVERNN_OK) return s;
  if (c.cond_dim > 0) {
    std::vector<float> wc((size_t)3 * H * c.cond_dim);
    for (size_t i = 0; i < wc.size(); ++i) wc[i] = rd(w->W_cond[i]);
    s = m->upload(&m->d_Wc, wc.data(), wc.size() * 4);
    if (s != WAVERNN_OK) return s;
  }
  HIPOK(hipFuncSetAttribute(wr_small_kernel_ptr(), hipFuncAttributeMaxDynamicSharedMemorySize, L.total_floats * 4));
  return WAVERNN_OK;
}

// One MFMA fragment (operand B of v_mfma_f32_16x16x32_bf16) of a matrix M(row, col):
// lane l holds row rowof(l % 16), columns col0 + 8*(l/16) .. +7, as bf16.
template <class M, class RowOf>
void frag(uint16_t* dst, M&& mat, RowOf&& rowof, int col0) {
  for (int l = 0; l < 64; ++l) {
    const int row = rowof(l % 16);
    for (int e = 0; e < 8; ++e) dst[l * 8 + e] = f2bf(mat(row, col0 + 8 * (l / 16) + e));
  }
}

// Head fragments: wave w of the head holding slice s holds O1 / O3 row tile
// RT s + w % RT over column tiles (w / RT) KH .. +KH, and O2 / O4 class tiles
// 2w, 2w+1 over the slice's HR columns (KO column tiles each).  Without split
// MLPs head j holds slice j as [O1][O3][O2][O4]; with them head j < NK holds
// [O1][O2] of slice j and head NK + j [O3][O4] of slice j.
std::vector<uint16_t> pack_heads(const PersistPlan& P, const wavernn_weights* w) {
  const int Hh = P.Hh, KH = P.KH, RT = P.RT, HR = P.HR, KO = P.KO;
  const bool split = P.NH == 2 * P.NK;
  auto O1m = [&](int r, int k) { return w->O1[(size_t)r * Hh + k]; };
  auto O3m = [&](int r, int k) { return w->O3[(size_t)r * Hh + k]; };
  auto O2m = [&](int v, int k) { return w->O2[(size_t)v * Hh + k]; };
  auto O4m = [&](int v, int k) { return w->O4[(size_t)v * Hh + k]; };
  std::vector<uint16_t> hw((size_t)P.NH * 8 * P.hw_frags * 512);
  for (int j = 0; j < P.NH; ++j)
    for (int wv = 0; wv < 8; ++wv) {
      uint16_t* d = hw.data() + (size_t)(j * 8 + wv) * P.hw_frags * 512;
      const int sl = j % P.NK;
      const int r0 = HR * sl + 16 * (wv % RT), k0 = 32 * (wv / RT) * KH;
      auto rows = [&](int r) { return r0 + r; };
      auto cls = [&](int i) { const int v0 = 16 * (2 * wv + i / KO); return [v0](int r) { return v0 + r; }; };
      if (split) {
        const bool fine = j >= P.NK;
        for (int i = 0; i < KH; ++i)
          fine ? frag(d + (size_t)i * 512, O3m, rows, k0 + 32 * i) : frag(d + (size_t)i * 512, O1m, rows, k0 + 32 * i);
        for (int i = 0; i < 2 * KO; ++i) {
          const int col = HR * sl + 32 * (i % KO);
          uint16_t* di = d + (size_t)(KH + i) * 512;
          fine ? frag(di, O4m, cls(i), col) : frag(di, O2m, cls(i), col);
        }
        continue;
      }
      for (int i = 0; i < KH; ++i) {
        frag(d + (size_t)i * 512, O1m, rows, k0 + 32 * i);
        frag(d + (size_t)(KH + i) * 512, O3m, rows, k0 + 32 * i);
      }
      for (int i = 0; i < 2 * KO; ++i) {
        const int col = HR * sl + 32 * (i % KO);
        frag(d + (size_t)(2 * KH + i) * 512, O2m, cls(i), col);
        frag(d + (size_t)(2 * KH + 2 * KO + i) * 512, O4m, cls(i), col);
      }
    }
  return hw;
}

// Arrays every persistent plan uses: head fragments, I*, biases, the
// conditioning projection, the per-frame table and the exchange words.
wavernn_status upload_common(wavernn_model* m, const wavernn_weights* w) {
  const wavernn_config& c = m->cfg;
  const PersistPlan& P = m->plan;
  const int H = P.H, Hh = P.Hh;
  Rounder rd{true};
  wavernn_status s;
  {
    std::vector<uint16_t> hw = pack_heads(P, w);
    if ((s = m->upload(&m->d_hw, hw.data(), hw.size() * 2)) != WAVERNN_OK) return s;
  }
  std::vector<float> Iv((size_t)9 * H), bv((size_t)3 * H);
  for (int row = 0; row < 3 * H; ++row) {
    for (int q = 0; q < 3; ++q) Iv[row * 3 + q] = (q == 2 && row % H < Hh) ? 0.0f : rd(w->I[row * 3 + q]);
    bv[row] = rd(w->b[row]);
  }
  std::vector<float> b1(Hh), b2(256), b3(Hh), b4(256);
  for (int k = 0; k < Hh; ++k) b1[k] = rd(w->b1[k]), b3[k] = rd(w->b3[k]);
  for (int v = 0; v < 256; ++v) b2[v] = rd(w->b2[v]), b4[v] = rd(w->b4[v]);
  if ((s = m->upload(&m->d_I, Iv.data(), Iv.size() * 4)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_bias, bv.data(), bv.size() * 4)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_b1, b1.data(), Hh * 4)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_b2, b2.data(), 256 * 4)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_b3, b3.data(), Hh * 4)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_b4, b4.data(), 256 * 4)) != WAVERNN_OK) return s;
  if (c.cond_dim > 0) {
    std::vector<float> wc((size_t)3 * H * c.cond_dim);
    for (size_t i = 0; i < wc.size(); ++i) wc[i] = rd(w->W_cond[i]);
    if ((s = m->upload(&m->d_Wc, wc.data(), wc.size() * 4)) != WAVERNN_OK) return s;
  }
  m->cb_cap = c.cond_dim > 0 ? 1024 : 1;
  if ((s = m->alloc(&m->d_cb, (size_t)m->cb_cap * 3 * H * 4)) != WAVERNN_OK) return s;
  if ((s = m->alloc(&m->d_xc, (size_t)(P.x_words + 1) / 2 * 8)) != WAVERNN_OK) return s;
  return WAVERNN_OK;
}

// The whole persistent grid must fit on the device at once.
wavernn_status check_coresident(wavernn_model* m, const void* k, int grid, int lds, const char* what) {
  HIPOK(hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, lds));
  int per_cu = 0;
  HIPOK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, WR_THREADS, lds));
  hipDeviceProp_t prop;
  HIPOK(hipGetDeviceProperties(&prop, m->device));
  if (per_cu < 1 || per_cu * prop.multiProcessorCount < grid)
    return fail(WAVERNN_E_UNSUPPORTED, "%s grid of %d workgroups cannot be co-resident (%d per CU, %d CUs)", what,
                grid, per_cu, prop.multiProcessorCount);
  return WAVERNN_OK;
}

int score_lds(int H);
int score_multi_lds(int H);

// Launch s of n persistent grids side by side: heads and mirrors on XCD
// 8 s / n, units spread over the XCDs.
PersistPlan fan_plan(const wavernn_model* m, int s, int n) {
  PersistPlan P = m->plan;
  wr_place(&P, 8 * s / n, 255);
  return P;
}

// Concurrent batch-1 launches for up to WR_FAN utterances, when that many
// persistent grids fit the device together: internal streams (default
// priority), fork / join events, and per-launch exchange words.
wavernn_status build_fanout(wavernn_model* m) {
  const PersistPlan& P = m->plan;
  int per_cu = 0;
  HIPOK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, m->pk, WR_THREADS, P.lds));
  hipDeviceProp_t prop;
  HIPOK(hipGetDeviceProperties(&prop, m->device));
  // launch i of n side by side puts its heads and mirrors on XCD 8 i / n and
  // spreads its units (fan_plan); n fits when every XCD holds the busy blocks
  // of all n grids at once (idle blocks return at once)
  int n = std::min(WR_FAN, (int)m->cfg.max_streams);
  for (; n >= 2; --n) {
    int busy[8] = {};
    for (int i = 0; i < n; ++i) {
      const PersistPlan Q = fan_plan(m, i, n);
      for (int b = 0; b < Q.grid; ++b)
        if (wr_role(Q, b) >= 0) ++busy[b % 8];
    }
    bool fits = per_cu >= 1;
    for (int x = 0; x < 8; ++x) fits = fits && busy[x] <= per_cu * (prop.multiProcessorCount / 8);
    if (fits) break;
  }
  if (n < 2) return WAVERNN_OK;
  HIPOK(hipEventCreateWithFlags(&m->fan_fork, hipEventDisableTiming));
  for (int i = 0; i < n; ++i) {
    if (i + 1 < n) {   // launch 0 runs on the caller's stream
      HIPOK(hipStreamCreateWithFlags(&m->fan_st[i], hipStreamNonBlocking));
      HIPOK(hipEventCreateWithFlags(&m->fan_join[i], hipEventDisableTiming));
    }
    wavernn_status s = m->alloc(&m->d_fxc[i], (size_t)(P.x_words + 1) / 2 * 8);
    if (s != WAVERNN_OK) return s;
  }
  m->nfan = n;
  if (m->sk) {   // the scoring recurrences' grids (H / 16 workgroups each) of n launches together
    const int H = P.H;
    int c1 = 0, c8 = 0;
    HIPOK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&c1, m->sk, WR_THREADS, score_lds(H)));
    if (m->smk) HIPOK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&c8, m->smk, WR_THREADS, score_multi_lds(H)));
    const int per_cu = m->smk ? std::min(c1, c8) : c1;
    m->score_fan = per_cu * prop.multiProcessorCount >= n * (H / 16);
  }
  return WAVERNN_OK;
}

// Dense unit workgroups of the persistent plan (R tiles in LDS and VGPRs).
wavernn_status upload_dense_units(wavernn_model* m, const wavernn_weights* w) {
  const PersistPlan& P = m->plan;
  const int H = P.H, Hh = P.Hh, KT = P.KT, UCT = P.UCT;
  REff R{&m->cfg, w};
  auto Rm = [&](int r, int k) { return R(r, k); };
  // units: R row of row tile `tile` of a half, lane row r
  auto rrow = [&](int tile, bool fine, int r) {
    const int g = tile / (Hh / 16), i = 16 * (tile % (Hh / 16)) + r;
    return g * H + (fine ? Hh : 0) + i;
  };
  // unit k's LDS block: [coarse tiles][KT] then [fine tiles][KT] fragments over
  // the coarse columns; ur: [coarse tiles | fine tiles][KT] over the fine columns
  const size_t NT = (size_t)P.NU * UCT;
  std::vector<uint16_t> uw((size_t)P.NU * P.u_lds_w / 2), ur(2 * NT * KT * 512);
  for (int k = 0; k < P.NU; ++k) {
    uint16_t* d = uw.data() + (size_t)k * P.u_lds_w / 2;
    for (int q = 0; q < UCT; ++q) {
      const int tile = k * UCT + q;
      for (int fine = 0; fine < 2; ++fine) {
        auto rows = [&](int r) { return rrow(tile, fine != 0, r); };
        for (int kt = 0; kt < KT; ++kt) {
          frag(d + (size_t)(fine * UCT * KT + q * KT + kt) * 512, Rm, rows, 32 * kt);
          frag(ur.data() + ((fine * NT + tile) * KT + kt) * 512, Rm, rows, Hh + 32 * kt);
        }
      }
    }
  }
  wavernn_status s;
  if ((s = m->upload(&m->d_uw, uw.data(), uw.size() * 2)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_ur, ur.data(), ur.size() * 2)) != WAVERNN_OK) return s;
  if (P.NM == 0) return WAVERNN_OK;
  // mirror j, wave w: coarse row tiles 12 j + 3 (w % 4) + r (r < 3) over the
  // fine column tiles (w / 4) MK + i (i < MK = KT / 2), as [r][i] fragments
  const int MK = KT / 2;
  std::vector<uint16_t> mw((size_t)P.NM * 8 * P.mw_frags * 512);
  for (int j = 0; j < P.NM; ++j)
    for (int wv = 0; wv < 8; ++wv) {
      uint16_t* d = mw.data() + (size_t)(j * 8 + wv) * P.mw_frags * 512;
      for (int r = 0; r < 3; ++r) {
        const int tile = WR_MTILES * j + 3 * (wv % 4) + r;
        auto rows = [&](int rr) { return rrow(tile, false, rr); };
        for (int i = 0; i < MK; ++i) frag(d + (size_t)(r * MK + i) * 512, Rm, rows, Hh + 32 * ((wv / 4) * MK + i));
      }
    }
  return m->upload(&m->d_mw, mw.data(), mw.size() * 2);
}

wavernn_status build_persist(wavernn_model* m, const wavernn_weights* w) {
  const PersistPlan& P = m->plan;
  m->pk = wr_persist_kernel_ptr(P.KH);
  if (!m->pk) return fail(WAVERNN_E_UNSUPPORTED, "hidden %d: no persistent kernel instantiation", P.H);
  wavernn_status s;
  if ((s = upload_dense_units(m, w)) != WAVERNN_OK) return s;
  if ((s = upload_common(m, w)) != WAVERNN_OK) return s;
  return check_coresident(m, m->pk, P.grid, P.lds, "persistent");
}

// Fused Subscale WaveRNN 2x (Sec. 4.4): the dense units of the batch-1 plan,
// fused heads (block-diagonal first layers and 64 nibble logits per half),
// I* with its six columns masked per quarter.  Head j, wave w holds O1 / O3
// rows 64 j + 16 (w % 4) over column chunk w / 4 (KH tiles), then class tile
// w (< 4) of the 64 nibble logits over the head's 64 columns.
wavernn_status build_fused(wavernn_model* m, const wavernn_weights* w) {
  const wavernn_config& c = m->cfg;
  PersistPlan& P = m->plan;
  const int H = P.H, Hh = P.Hh, Q = Hh / 2, KH = P.KH, KO = P.KO;
  m->pk = wr_fused_kernel_ptr(KH);
  if (!m->pk) return fail(WAVERNN_E_UNSUPPORTED, "hidden %d: no fused kernel instantiation", H);
  wavernn_status s;
  if ((s = upload_dense_units(m, w)) != WAVERNN_OK) return s;
  // first layer of the half at level lv (Hh x Hh, block diagonal) and its 64 nibble-logit rows
  auto O1f = [&](int lv) {
    return [=](int r, int k) {
      return r / Q == k / Q ? w->O1[((size_t)(2 * lv + r / Q) * Q + r % Q) * Q + k % Q] : 0.0f;
    };
  };
  auto O2f = [&](int lv) {
    return [=](int v, int k) {   // v = 32 s + 16 part + nibble
      const int sv = v / 32;
      return sv == k / Q ? w->O2[((size_t)((2 * lv + sv) * 2 + (v / 16) % 2) * 16 + v % 16) * Q + k % Q] : 0.0f;
    };
  };
  std::vector<uint16_t> hw((size_t)P.NH * 8 * P.hw_frags * 512, 0);
  for (int j = 0; j < P.NH; ++j)
    for (int wv = 0; wv < 8; ++wv) {
      uint16_t* d = hw.data() + (size_t)(j * 8 + wv) * P.hw_frags * 512;
      const int r0 = 64 * j + 16 * (wv % 4), k0 = 32 * (wv / 4) * KH;
      auto rows = [&](int r) { return r0 + r; };
      for (int i = 0; i < KH; ++i) {
        frag(d + (size_t)i * 512, O1f(0), rows, k0 + 32 * i);
        frag(d + (size_t)(KH + i) * 512, O1f(1), rows, k0 + 32 * i);
      }
      if (wv >= 4) continue;
      auto cls = [&](int r) { return 16 * wv + r; };
      for (int kt = 0; kt < KO; ++kt) {
        frag(d + (size_t)(2 * KH + kt) * 512, O2f(0), cls, 64 * j + 32 * kt);
        frag(d + (size_t)(2 * KH + KO + kt) * 512, O2f(1), cls, 64 * j + 32 * kt);
      }
    }
  if ((s = m->upload(&m->d_hw, hw.data(), hw.size() * 2)) != WAVERNN_OK) return s;
  Rounder rd{true};
  std::vector<float> Iv((size_t)18 * H), bv((size_t)3 * H);
  for (int row = 0; row < 3 * H; ++row) {
    const int i = row % H;
    for (int q = 0; q < 6; ++q) {
      const bool keep = q < 4 || (i >= Hh && q == 4 + (i - Hh) / Q);   // the I* mask per quarter
      Iv[(size_t)row * 6 + q] = keep ? rd(w->I[(size_t)row * 6 + q]) : 0.0f;
    }
    bv[row] = rd(w->b[row]);
  }
  std::vector<float> b1(2 * Hh), b2(128);
  for (int k = 0; k < 2 * Hh; ++k) b1[k] = rd(w->b1[k]);   // [level][s][Q]: coarse half, then fine half
  for (int v = 0; v < 128; ++v) b2[v] = rd(w->b2[v]);      // [level][s][part][16]
  if ((s = m->upload(&m->d_I, Iv.data(), Iv.size() * 4)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_bias, bv.data(), bv.size() * 4)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_b1, b1.data(), b1.size() * 4)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_b2, b2.data(), b2.size() * 4)) != WAVERNN_OK) return s;
  m->d_b3 = m->d_b1 + Hh;
  m->d_b4 = m->d_b2 + 64;
  if (c.cond_dim > 0) {
    std::vector<float> wc((size_t)3 * H * c.cond_dim);
    for (size_t i = 0; i < wc.size(); ++i) wc[i] = rd(w->W_cond[i]);
    if ((s = m->upload(&m->d_Wc, wc.data(), wc.size() * 4)) != WAVERNN_OK) return s;
  }
  m->cb_cap = c.cond_dim > 0 ? 1024 : 1;
  if ((s = m->alloc(&m->d_cb, (size_t)m->cb_cap * 3 * H * 4)) != WAVERNN_OK) return s;
  if ((s = m->alloc(&m->d_xc, (size_t)(P.x_words + 1) / 2 * 8)) != WAVERNN_OK) return s;
  m->fused = true;
  return check_coresident(m, m->pk, P.grid, P.lds, "fused");
}

// Block-sparse R (Sec. 3.2) as the block-sparse units store it (layout in
// sparse_plan): per unit and half of the columns, the kept blocks of each
// block-row dealt to the SL parts of its rows in turn, one u16 block-column
// index per kept block, and each lane's row of the block's weights.  Rows per
// unit SR is the first of 32, 64, 128, 16 whose blocks fit LDS and whose grid
// fits (fewer rows per unit: shorter walks on the way to the heads).
wavernn_status build_sparse(wavernn_model* m, const wavernn_weights* w) {
  const wavernn_config& c = m->cfg;
  const int H = c.hidden, Hh = H / 2;
  const int bh = c.r_format == WAVERNN_R_BSR_4X4 ? 4 : 16, bw = c.r_format == WAVERNN_R_BSR_4X4 ? 4 : 1;
  // kept block columns of every block-row (gate g, block-row i / bh), coarse and fine columns apart
  const int nbr = 3 * H / bh;
  std::vector<std::vector<uint16_t>> kept((size_t)2 * nbr);
  for (int r = 0; r < nbr; ++r) {
    const uint8_t* mrow = w->R_block_mask + (size_t)r * (H / bw);
    for (int bc = 0; bc < H / bw; ++bc)
      if (mrow[bc]) kept[(size_t)2 * r + (bc * bw >= Hh)].push_back((uint16_t)(bc * bw));
  }
  hipDeviceProp_t prop;
  HIPOK(hipGetDeviceProperties(&prop, m->device));
  PersistPlan& P = m->plan;
  bool ok = false;
  for (int SR : {32, 64, 128, 16}) {
    const int SL = 256 / SR;
    size_t nb[2] = {1, 1};   // longest part list per half
    for (size_t q = 0; q < kept.size(); ++q) nb[q & 1] = std::max(nb[q & 1], (kept[q].size() + SL - 1) / SL);
    if (sparse_plan(H, SR, bh, bw, (int)nb[0], (int)nb[1], &P) && P.grid <= prop.multiProcessorCount) {
      ok = true;
      break;
    }
  }
  if (!ok) return fail(WAVERNN_E_UNSUPPORTED, "hidden %d: the kept blocks of R do not fit a block-sparse plan", H);
  m->pk = wr_sparse_kernel_ptr(P.KH, P.GU);
  if (!m->pk) return fail(WAVERNN_E_UNSUPPORTED, "hidden %d: no block-sparse kernel instantiation", H);
  const int NR = P.NRC + P.NRF, SL = P.SL, BR = P.BR;
  const size_t per = (size_t)P.u_lds_w / 2;            // u16 per unit block
  std::vector<uint16_t> img((size_t)P.NU * per, 0);
  for (int k = 0; k < P.NU; ++k) {
    uint16_t* wt = img.data() + (size_t)k * per;               // [NR][256] x (4 or 1) bf16
    uint16_t* ix = wt + P.u_wb / 2;                            // [NR][BR][SL]
    for (int ph = 0; ph < 2; ++ph) {
      const int nr = ph ? P.NRF : P.NRC, r0 = ph ? P.NRC : 0;
      for (int R = 0; R < BR; ++R) {
        const int br = (P.SR * k) / bh + R;                    // block-row over the stacked gates
        const std::vector<uint16_t>& L = kept[(size_t)2 * br + ph];
        for (int part = 0; part < SL; ++part)
          for (int sl = 0; sl < nr; ++sl) {
            const size_t b = (size_t)part + (size_t)SL * sl;   // this part's sl-th block of the block-row
            const bool real = b < L.size();
            const int col0 = real ? L[b] : (ph ? Hh : 0);
            const int slot = r0 + sl, qd = slot / 4, qe = slot % 4;   // 16 x 1: quads of slots
            if (bw == 4) ix[((size_t)slot * BR + R) * SL + part] = (uint16_t)col0;
            else ix[(((size_t)qd * BR + R) * SL + part) * 4 + qe] = (uint16_t)col0;
            for (int rb = 0; rb < bh; ++rb) {                  // the block-row's rows: lanes (R bh + rb) SL + part
              const int lane = (R * bh + rb) * SL + part;
              const int row = P.SR * k + R * bh + rb;
              if (bw == 4) {
                for (int e = 0; e < 4; ++e)
                  wt[((size_t)slot * 256 + lane) * 4 + e] = real ? f2bf(w->R[(size_t)row * H + col0 + e]) : 0;
              } else {
                wt[((size_t)qd * 256 + lane) * 4 + qe] = real ? f2bf(w->R[(size_t)row * H + col0]) : 0;
              }
            }
          }
      }
    }
  }
  wavernn_status s;
  if ((s = m->upload(&m->d_uw, img.data(), img.size() * 2)) != WAVERNN_OK) return s;
  if ((s = upload_common(m, w)) != WAVERNN_OK) return s;
  m->sparse = true;
  (void)NR;
  return check_coresident(m, m->pk, P.grid, P.lds, "block-sparse");
}

// Batched path: unit blocks for WR_BUCT = 4 row tiles per half (the head
// fragments are the batch-1 ones).
wavernn_status build_batch(wavernn_model* m, const wavernn_weights* w) {
  const BatchPlan& B = m->bplan;
  const int H = B.H, Hh = B.Hh, KT = B.KT;
  REff R{&m->cfg, w};
  auto frag = [&](uint16_t* dst, int tile, bool fine, int col0) {
    for (int l = 0; l < 64; ++l) {
      const int g = tile / (Hh / 16), i = 16 * (tile % (Hh / 16)) + l % 16;
      const int row = g * H + (fine ? Hh : 0) + i;
      for (int e = 0; e < 8; ++e) dst[l * 8 + e] = f2bf(R(row, col0 + 8 * (l / 16) + e));
    }
  };
  std::vector<uint16_t> uw((size_t)B.NU * B.u_lds_w / 2), ur((size_t)B.NU * 8 * KT * 512);
  for (int k = 0; k < B.NU; ++k) {
    uint16_t* d = uw.data() + (size_t)k * B.u_lds_w / 2;
    for (int q = 0; q < WR_BUCT; ++q) {
      const int tile = k * WR_BUCT + q;
      for (int kt = 0; kt < KT; ++kt) {
        frag(d + (size_t)(q * KT + kt) * 512, tile, false, 32 * kt);                        // coarse tile, coarse cols
        frag(d + (size_t)((WR_BUCT + q) * KT + kt) * 512, tile, true, Hh + 32 * kt);         // fine tile, fine cols
        frag(ur.data() + ((size_t)(k * 8 + q) * KT + kt) * 512, tile, false, Hh + 32 * kt);  // coarse tile, fine cols
        frag(ur.data() + ((size_t)(k * 8 + 4 + q) * KT + kt) * 512, tile, true, 32 * kt);    // fine tile, coarse cols
      }
    }
  }
  wavernn_status s;
  if (B.KX > 0) {   // context projection W_ctx: [unit][wave][column tile] fragments of the wave's row tile
    const int Dx = m->cfg.ctx_dim;
    std::vector<uint16_t> ux((size_t)B.NU * 8 * B.KX * 512);
    for (int k = 0; k < B.NU; ++k)
      for (int wv = 0; wv < 8; ++wv) {
        const int tile = k * WR_BUCT + (wv & 3);
        const bool fine = wv >= 4;
        for (int kt = 0; kt < B.KX; ++kt) {
          uint16_t* d = ux.data() + ((size_t)(k * 8 + wv) * B.KX + kt) * 512;
          for (int l = 0; l < 64; ++l) {
            const int g = tile / (Hh / 16), i = 16 * (tile % (Hh / 16)) + l % 16;
            const int row = g * H + (fine ? Hh : 0) + i;
            for (int e = 0; e < 8; ++e) d[l * 8 + e] = f2bf(w->W_ctx[(size_t)row * Dx + 32 * kt + 8 * (l / 16) + e]);
          }
        }
      }
    if ((s = m->upload(&m->d_bux, ux.data(), ux.size() * 2)) != WAVERNN_OK) return s;
  }
  if ((s = m->upload(&m->d_buw, uw.data(), uw.size() * 2)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_bur, ur.data(), ur.size() * 2)) != WAVERNN_OK) return s;
  // every plan a call may use (2 vectors per group up to 16 vectors, 4 up to
  // 32, 8 above): the largest grid of each group size must fit, and the
  // exchange buffer holds the largest of them
  const int maxv = m->cfg.max_streams * m->cfg.subscale;
  size_t xwords = 0;
  for (int v : {std::min(maxv, 2 * WR_BL), std::min(maxv, 4 * WR_BL), maxv}) {
    BatchPlan Q;
    if (!batch_plan(H, v, &Q, m->cfg.ctx_dim, m->cfg.subscale, horizon_of(m->cfg), lead_of(m->cfg), m->has_cnn))
      return fail(WAVERNN_E_UNSUPPORTED, "no batched plan for %d vectors (future horizon %d: sample ring of the "
                  "units too large for LDS?)", v, horizon_of(m->cfg));
    const void* k = wr_batch_kernel_ptr(Q.KH, Q.KX > 0, Q.L, horizon_of(m->cfg) >= 0);
    if (!k) return fail(WAVERNN_E_UNSUPPORTED, "hidden %d: no batched kernel instantiation", H);
    if ((s = check_coresident(m, k, Q.grid, Q.lds, "batched")) != WAVERNN_OK) return s;
    xwords = std::max(xwords, (size_t)Q.G * Q.x_words);
  }
  if ((s = m->alloc(&m->d_bxc, (xwords + 1) / 2 * 8)) != WAVERNN_OK) return s;
  m->has_batch = true;
  return WAVERNN_OK;
}

// Fragments [N / 16][K / 32] (operand B of v_mfma_f32_16x16x32_bf16) of a
// matrix W(n, k), n < N, k < K (K a multiple of 32), bf16 round to nearest even.
template <class M>
void pack_gemm(std::vector<uint16_t>& dst, M&& mat, int N, int K) {
  const size_t base = dst.size();
  dst.resize(base + (size_t)N * K);
  for (int nt = 0; nt < N / 16; ++nt)
    for (int kt = 0; kt < K / 32; ++kt)
      frag(dst.data() + base + ((size_t)nt * (K / 32) + kt) * 512, mat, [&](int r) { return 16 * nt + r; }, 32 * kt);
}

// Rows a conditioning CNN of `layers` layers sees past its own row: each layer
// reaches 2 d further, d = 2^(l mod 5) (124 for ten layers).
int cnn_reach(int layers) {
  int r = 0;
  for (int l = 0; l < layers; ++l) r += 2 << (l % 5);
  return r;
}

// Grow the context table to `floats` (waits for `st` first when it has work that may read the old one).
wavernn_status grow_ctab(wavernn_model* m, size_t floats, hipStream_t* st) {
  if (floats <= (size_t)m->ctab_cap) return WAVERNN_OK;
  if (st) HIPOK(hipStreamSynchronize(*st));
  float* p = nullptr;
  wavernn_status s = m->alloc(&p, floats * 4);
  if (s != WAVERNN_OK) return s;
  // zeroed: a sampling chunk writes only the blocks of the sub-tensors it
  // runs, and idle lanes read (and discard) the others
  if (st) HIPOK(hipMemsetAsync(p, 0, floats * 4, *st));
  else HIPOK(hipMemset(p, 0, floats * 4));
  m->d_ctab = p;
  m->ctab_cap = (int64_t)floats;
  return WAVERNN_OK;
}

// The conditioning CNN's weights as GEMM fragments (input layer with its 2B
// columns padded to kin, then per layer convolution [Cc][3 Rc] and projection
// [Rc][Cc], then the output layer [Dx][Rc]) and biases.
wavernn_status build_cnn(wavernn_model* m, const wavernn_ctx_cnn* n) {
  auto& C = m->cnn;
  const int B = m->cfg.subscale, Dx = m->cfg.ctx_dim;
  C.Rc = n->res_channels;
  C.Cc = n->conv_channels;
  C.layers = n->layers;
  C.kin = (2 * B + 31) / 32 * 32;
  const int Rc = C.Rc, Cc = C.Cc, kin = C.kin;
  Rounder rd{true};
  std::vector<uint16_t> w;
  std::vector<float> b;
  auto mark = [&]() {
    C.woff.push_back(w.size() / 8);
    C.boff.push_back(b.size());
  };
  mark();
  pack_gemm(w, [&](int o, int q) { return q < 2 * B ? n->Win[(size_t)o * 2 * B + q] : 0.0f; }, Rc, kin);
  for (int o = 0; o < Rc; ++o) b.push_back(rd(n->bin[o]));
  for (int l = 0; l < C.layers; ++l) {
    mark();
    const float* Wc = n->Wc + (size_t)l * Cc * 3 * Rc;
    pack_gemm(w, [&](int c, int q) { return Wc[(size_t)c * 3 * Rc + q]; }, Cc, 3 * Rc);
    for (int c = 0; c < Cc; ++c) b.push_back(rd(n->bc[(size_t)l * Cc + c]));
    mark();
    const float* Wo = n->Wo + (size_t)l * Rc * Cc;
    pack_gemm(w, [&](int o, int c) { return Wo[(size_t)o * Cc + c]; }, Rc, Cc);
    for (int o = 0; o < Rc; ++o) b.push_back(rd(n->bo[(size_t)l * Rc + o]));
  }
  mark();
  pack_gemm(w, [&](int o, int q) { return n->Wp[(size_t)o * Rc + q]; }, Dx, Rc);
  for (int o = 0; o < Dx; ++o) b.push_back(rd(n->bp[o]));
  wavernn_status s;
  if ((s = m->upload(&C.w, w.data(), w.size() * 2)) != WAVERNN_OK) return s;
  if ((s = m->upload(&C.bias, b.data(), b.size() * 4)) != WAVERNN_OK) return s;
  HIPOK(hipFuncSetAttribute(wr_cnn_gemm_ptr(), hipFuncAttributeMaxDynamicSharedMemorySize, 2 * CNN_LDS_BUF));
  m->has_cnn = true;
  return WAVERNN_OK;
}

// LDS of the scoring recurrence: the operand image of h, [3][16] pre-activations, misc.
int score_lds(int H) { return H / 32 * WR_FRAG + 48 * 4 + 64; }
int score_multi_lds(int H) { return H / 32 * WR_FRAG + 3 * 8 * 16 * 4 + 64; }

// Teacher-forced scoring on the dense batch-1 plan: the recurrence kernel
// (the plan's units, heads that evaluate their own slices from the given
// bytes) and the output layers as GEMM fragments for the matrix cores: O1 and
// O3 with their rows padded to NP = Hh rounded up to 128, O2 and O4 with their
// columns padded to NP, biases rounded like the sampling heads' and padded
// with zeros (a padded first-layer row is relu(0) = 0 and meets a zero column).
wavernn_status build_score(wavernn_model* m, const wavernn_weights* w) {
  const PersistPlan& P = m->plan;
  const int H = P.H, Hh = P.Hh, NP = (Hh + 127) / 128 * 128, KT2 = H / 32;
  m->sk = wr_score_kernel_ptr(KT2);
  if (!m->sk) return fail(WAVERNN_E_UNSUPPORTED, "hidden %d: no scoring kernel instantiation", H);
  {   // recurrence: workgroup k, gate g holds rows g H + 16 k .. + 15 over every column tile
    REff R{&m->cfg, w};
    auto Rm = [&](int r, int c) { return R(r, c); };
    std::vector<uint16_t> rw((size_t)H / 16 * 3 * KT2 * 512);
    for (int k = 0; k < H / 16; ++k)
      for (int g = 0; g < 3; ++g)
        for (int kt = 0; kt < KT2; ++kt)
          frag(rw.data() + ((size_t)(k * 3 + g) * KT2 + kt) * 512, Rm, [&](int r) { return g * H + 16 * k + r; },
               32 * kt);
    wavernn_status s = m->upload(&m->d_srw, rw.data(), rw.size() * 2);
    if (s != WAVERNN_OK) return s;
  }
  Rounder rd{m->cfg.weight_dtype == WAVERNN_BF16};
  std::vector<uint16_t> wv;
  std::vector<float> bv;
  const float* Os[4] = {w->O1, w->O2, w->O3, w->O4};
  const float* bs[4] = {w->b1, w->b2, w->b3, w->b4};
  for (int k = 0; k < 4; ++k) {
    m->sw_off[k] = wv.size() / 8;
    m->sb_off[k] = bv.size();
    const float* O = Os[k];
    if (k % 2 == 0) {
      pack_gemm(wv, [&](int o, int q) { return o < Hh ? O[(size_t)o * Hh + q] : 0.0f; }, NP, Hh);
      for (int o = 0; o < NP; ++o) bv.push_back(o < Hh ? rd(bs[k][o]) : 0.0f);
    } else {
      pack_gemm(wv, [&](int o, int q) { return q < Hh ? O[(size_t)o * Hh + q] : 0.0f; }, 256, NP);
      for (int o = 0; o < 256; ++o) bv.push_back(rd(bs[k][o]));
    }
  }
  m->sc_np = NP;
  wavernn_status s;
  if ((s = m->upload(&m->d_sw, wv.data(), wv.size() * 2)) != WAVERNN_OK) return s;
  if ((s = m->upload(&m->d_sb, bv.data(), bv.size() * 4)) != WAVERNN_OK) return s;
  HIPOK(hipFuncSetAttribute(wr_cnn_gemm_ptr(), hipFuncAttributeMaxDynamicSharedMemorySize, 2 * CNN_LDS_BUF));
  if ((s = check_coresident(m, m->sk, H / 16, score_lds(H), "scoring")) != WAVERNN_OK) return s;
  // several utterances per launch where its grid fits too (else one at a time)
  m->smk = wr_score_multi_ptr(H / 32);
  if (m->smk && check_coresident(m, m->smk, H / 16, score_multi_lds(H), "scoring") != WAVERNN_OK) m->smk = nullptr;
  return WAVERNN_OK;
}

// One CNN layer as a GEMM (see CnnGemmArgs).
struct CnnRows {   // which utterance rows the blocks of a CNN run cover
  int B;
  int64_t row0, row_step, rows_utt;
};

// A CNN GEMM's K loop sums in groups of CNN_GROUP K-steps (always, so that results
// never depend on the rows of a run); a GEMM with fewer tiles than CUs runs
// each group on its own workgroup and adds them in wr_cnn_reduce.
#define CNN_GROUP 6
int cnn_split(int M, int N, int K) {
  const int tiles = (M + CNN_TM - 1) / CNN_TM * (N / CNN_TN), groups = (K / 32 + CNN_GROUP - 1) / CNN_GROUP;
  return tiles < 256 && groups > 1 ? groups : 1;
}

// A streamed run's rows (see CnnGemmArgs::rng): sub-tensor s's run rows are its utterance rows
// lo[s] .. hi[s] - 1; whole-utterance source and destination arrays where src_abs / dst_abs.
struct CnnRng {
  const int* lo;
  const int* hi;
  int src_abs, dst_abs;
};

wavernn_status cnn_gemm(const float* src, int kin, int taps, int dil, int rows, const CnnRows& cr, int M,
                        const uint4* w, const float* bias, int N, float* dst, int epi, hipStream_t st,
                        float* part = nullptr, int out_B = 0, int out_s0 = 0, const CnnRng* rng = nullptr) {
  CnnGemmArgs g;
  memset(&g, 0, sizeof g);
  if (rng) {
    g.rng = 1;
    g.src_abs = rng->src_abs;
    g.dst_abs = rng->dst_abs;
    for (int s = 0; s < WR_CNN_MAXB; ++s) g.lo[s] = rng->lo[s], g.hi[s] = rng->hi[s];
  }
  g.src = src;
  g.kin = kin;
  g.taps = taps;
  g.dil = dil;
  g.rows = rows;
  g.B = cr.B;
  g.row0 = cr.row0;
  g.row_step = cr.row_step;
  g.rows_utt = cr.rows_utt;
  g.M = M;
  g.K = taps * kin;
  g.w = w;
  g.bias = bias;
  g.N = N;
  g.dst = dst;
  g.out_B = out_B ? out_B : cr.B;
  g.out_s0 = out_s0;
  g.epi = epi;
  g.group = CNN_GROUP;
  g.split = part ? cnn_split(M, N, g.K) : 1;
  g.part = part;
  g.tiles_m = (M + CNN_TM - 1) / CNN_TM;
  g.tiles = g.tiles_m * (N / CNN_TN);
  g.per_xcd = (g.tiles * g.split + 7) / 8;
  void* args[] = {&g};
  HIPOK(hipLaunchKernel(wr_cnn_gemm_ptr(), dim3(8 * g.per_xcd), dim3(CNN_THREADS), args, 2 * CNN_LDS_BUF, st));
  if (g.split > 1)
    HIPOK(hipLaunchKernel(wr_cnn_reduce_ptr(), dim3((unsigned)(((int64_t)M * N + 255) / 256)), dim3(256), args, 0, st));
  return WAVERNN_OK;
}

// The conditioning CNN over windows of `win` rows per (utterance, sub-tensor),
// for the sub-tensors s0 .. s0 + nsb - 1: block (u, s) covers utterance rows
// row0 + s row_step .. + win - 1, samples of sub-tensor z counted up to row
// front0 + z front_step; out [U][B][win][Dx] (the other sub-tensors' blocks
// are left as they are).
wavernn_status run_cnn(wavernn_model* m, int U, const uint16_t* seq, int64_t n_samples, int win, int64_t row0,
                       int64_t row_step, int64_t front0, int64_t front_step, float* out, hipStream_t st, int s0 = 0,
                       int nsb = 0) {
  auto& C = m->cnn;
  const int B = m->cfg.subscale, Dx = m->cfg.ctx_dim;
  if (nsb <= 0) nsb = B;
  const int64_t M64 = (int64_t)U * nsb * win;
  if (M64 > (1 << 28)) return fail(WAVERNN_E_INVALID, "conditioning CNN: %lld rows, above 2^28", (long long)M64);
  const int M = (int)M64;
  if (M > C.cap) {   // grow the activations (an allocation: only when a call needs more rows than any before)
    HIPOK(hipStreamSynchronize(st));
    wavernn_status s;
    if ((s = m->alloc(&C.x, (size_t)M * C.kin * 4)) != WAVERNN_OK) return s;
    if ((s = m->alloc(&C.r, (size_t)M * C.Rc * 4)) != WAVERNN_OK) return s;
    if ((s = m->alloc(&C.act, (size_t)M * C.Cc * 4)) != WAVERNN_OK) return s;
    C.cap = M;
  }
  {   // the split GEMMs' partial products (the largest of the run's layers)
    int64_t need = 0;
    const int KN[4][2] = {{C.kin, C.Rc}, {3 * C.Rc, C.Cc}, {C.Cc, C.Rc}, {C.Rc, Dx}};
    for (auto& kn : KN) {
      const int sp = cnn_split(M, kn[1], kn[0]);
      if (sp > 1) need = std::max(need, (int64_t)sp * M * kn[1]);
    }
    if (need > C.part_cap) {
      HIPOK(hipStreamSynchronize(st));
      wavernn_status s;
      if ((s = m->alloc(&C.part, (size_t)need * 4)) != WAVERNN_OK) return s;
      C.part_cap = need;
    }
  }
  CnnInputArgs in;
  memset(&in, 0, sizeof in);
  in.seq = seq;
  in.n_samples = n_samples;
  in.B = B;
  in.rows = n_samples / B;
  in.win = win;
  in.row0 = row0;
  in.row_step = row_step;
  in.front0 = front0;
  in.front_step = front_step;
  in.s0 = s0;
  in.nsb = nsb;
  in.M = M;
  in.kin = C.kin;
  in.x = C.x;
  void* args[] = {&in};
  const int64_t nx = (int64_t)M * C.kin;
  HIPOK(hipLaunchKernel(wr_cnn_input_ptr(), dim3((unsigned)((nx + 255) / 256)), dim3(256), args, 0, st));
  wavernn_status s;
  size_t i = 0;
  const CnnRows cr{nsb, row0 + s0 * row_step, row_step, n_samples / B};
  if ((s = cnn_gemm(C.x, C.kin, 1, 0, win, cr, M, C.w + C.woff[i], C.bias + C.boff[i], C.Rc, C.r, 0, st, C.part)) !=
      WAVERNN_OK)
    return s;
  ++i;
  for (int l = 0; l < C.layers; ++l, i += 2) {
    if ((s = cnn_gemm(C.r, C.Rc, 3, 1 << (l % 5), win, cr, M, C.w + C.woff[i], C.bias + C.boff[i], C.Cc, C.act, 1,
                      st, C.part)) != WAVERNN_OK)
      return s;
    if ((s = cnn_gemm(C.act, C.Cc, 1, 0, win, cr, M, C.w + C.woff[i + 1], C.bias + C.boff[i + 1], C.Rc, C.r, 2,
                      st, C.part)) != WAVERNN_OK)
      return s;
  }
  return cnn_gemm(C.r, C.Rc, 1, 0, win, cr, M, C.w + C.woff[i], C.bias + C.boff[i], Dx, out, 0, st, C.part, B, s0);
}

// The conditioning CNN streamed over a sampling call (Sec. 4.2: the
// conditioning runs ahead of the sampler).  Level 0 is the input layer,
// levels 1 .. L the dilated layers, level L + 1 the output layer; before the
// chunk that starts at step t0, level v of sub-tensor s is final below row
// cnn_front(v, s, t0): the input rows of s hold the samples of the sub-tensors
// z < s, made below row t0 - z (F + 1), and a level-v row reads input rows up
// to its reach.  Each chunk computes every level's newly final rows once (from
// lo[v][s], then lo[v][s] = the front), the dilated layers in place in a
// whole-utterance residual array (a layer's convolution reads every row it
// needs before its projection updates any), and writes the output rows into
// the whole-utterance context table out [U][B][rows][Dx].  A row is computed
// with the arithmetic of a windowed run, so the table, and the samples, do not
// depend on the chunking.
int64_t cnn_front(const int* reach, int v, int s, int64_t t0, int F, int64_t rows) {
  int64_t f0 = t0 - (int64_t)(s - 1) * (F + 1);   // rows below f0: made by sub-tensor s - 1 (and so every z < s)
  if (f0 >= rows) return rows;                      // (past the utterance the taps are zero: final too)
  if (f0 < 0) f0 = 0;
  const int64_t f = f0 - reach[v];
  return f > 0 ? f : 0;
}

wavernn_status run_cnn_stream(wavernn_model* m, int U, const uint16_t* seq, int64_t n_samples, int64_t t0, int F,
                              int (*lo)[WR_CNN_MAXB], float* out, hipStream_t st) {
  auto& C = m->cnn;
  const int B = m->cfg.subscale, Dx = m->cfg.ctx_dim, L = C.layers;
  const int64_t rows = n_samples / B;
  int reach[2 * 32 + 2];
  reach[0] = 0;
  for (int l = 1; l <= L; ++l) reach[l] = reach[l - 1] + (2 << ((l - 1) % 5));
  reach[L + 1] = reach[L];
  // the whole-utterance residual array (an allocation only when a call needs more rows than any before)
  const int64_t rf = (int64_t)U * B * rows * C.Rc;
  if (rf > C.rfull_cap) {
    HIPOK(hipStreamSynchronize(st));
    wavernn_status s;
    if ((s = m->alloc(&C.rfull, (size_t)rf * 4)) != WAVERNN_OK) return s;
    C.rfull_cap = rf;
  }
  for (int v = 0; v <= L + 1; ++v) {
    int hi[WR_CNN_MAXB] = {}, a = -1, b = -1, n = 0;
    for (int s = 0; s < B; ++s) {
      hi[s] = (int)cnn_front(reach, v, s, t0, F, rows);
      if (hi[s] < lo[v][s]) hi[s] = lo[v][s];
      if (hi[s] > lo[v][s]) {
        if (a < 0) a = s;
        b = s;
        n = std::max(n, hi[s] - lo[v][s]);
      }
    }
    if (a < 0) continue;
    const int nsb = b - a + 1;
    const int64_t M64 = (int64_t)U * nsb * n;
    if (M64 > (1 << 28)) return fail(WAVERNN_E_INVALID, "conditioning CNN: %lld rows, above 2^28", (long long)M64);
    const int M = (int)M64;
    if (M > C.cap) {   // the run's transient rows
      HIPOK(hipStreamSynchronize(st));
      wavernn_status s;
      if ((s = m->alloc(&C.x, (size_t)M * C.kin * 4)) != WAVERNN_OK) return s;
      if ((s = m->alloc(&C.r, (size_t)M * C.Rc * 4)) != WAVERNN_OK) return s;
      if ((s = m->alloc(&C.act, (size_t)M * C.Cc * 4)) != WAVERNN_OK) return s;
      C.cap = M;
    }
    {
      int64_t need = 0;
      const int KN[4][2] = {{C.kin, C.Rc}, {3 * C.Rc, C.Cc}, {C.Cc, C.Rc}, {C.Rc, Dx}};
      for (auto& kn : KN) {
        const int sp = cnn_split(M, kn[1], kn[0]);
        if (sp > 1) need = std::max(need, (int64_t)sp * M * kn[1]);
      }
      if (need > C.part_cap) {
        HIPOK(hipStreamSynchronize(st));
        wavernn_status s;
        if ((s = m->alloc(&C.part, (size_t)need * 4)) != WAVERNN_OK) return s;
        C.part_cap = need;
      }
    }
    const CnnRows cr{nsb, 0, 0, rows};
    wavernn_status s;
    if (v == 0) {   // input rows, then r = Win x + bin into the residual array
      CnnInputArgs in;
      memset(&in, 0, sizeof in);
      in.seq = seq;
      in.n_samples = n_samples;
      in.B = B;
      in.rows = rows;
      in.win = n;
      in.front0 = t0 - 1;
      in.front_step = -(int64_t)(F + 1);
      in.s0 = a;
      in.nsb = nsb;
      in.M = M;
      in.kin = C.kin;
      in.x = C.x;
      in.rng = 1;
      for (int z = 0; z < WR_CNN_MAXB; ++z) in.lo[z] = lo[0][z];
      void* args[] = {&in};
      const int64_t nx = (int64_t)M * C.kin;
      HIPOK(hipLaunchKernel(wr_cnn_input_ptr(), dim3((unsigned)((nx + 255) / 256)), dim3(256), args, 0, st));
      const CnnRng rg{lo[0], hi, 0, 1};
      if ((s = cnn_gemm(C.x, C.kin, 1, 0, n, cr, M, C.w + C.woff[0], C.bias + C.boff[0], C.Rc, C.rfull, 0, st,
                        C.part, B, a, &rg)) != WAVERNN_OK)
        return s;
    } else if (v <= L) {   // layer v: convolution from the residual array, projection added back into it
      const size_t i = 1 + 2 * (size_t)(v - 1);
      const CnnRng conv{lo[v], hi, 1, 0}, proj{lo[v], hi, 0, 1};
      if ((s = cnn_gemm(C.rfull, C.Rc, 3, 1 << ((v - 1) % 5), n, cr, M, C.w + C.woff[i], C.bias + C.boff[i], C.Cc,
                        C.act, 1, st, C.part, B, a, &conv)) != WAVERNN_OK)
        return s;
      if ((s = cnn_gemm(C.act, C.Cc, 1, 0, n, cr, M, C.w + C.woff[i + 1], C.bias + C.boff[i + 1], C.Rc, C.rfull, 2,
                        st, C.part, B, a, &proj)) != WAVERNN_OK)
        return s;
    } else {   // output rows into the whole-utterance table
      const size_t i = 1 + 2 * (size_t)L;
      const CnnRng o{lo[v], hi, 1, 1};
      if ((s = cnn_gemm(C.rfull, C.Rc, 1, 0, n, cr, M, C.w + C.woff[i], C.bias + C.boff[i], Dx, out, 0, st, C.part,
                        B, a, &o)) != WAVERNN_OK)
        return s;
    }
    for (int z = 0; z < B; ++z) lo[v][z] = hi[z];
  }
  return WAVERNN_OK;
}

// Bias + conditioning table cb[s][f][3H] for n_streams streams of n_frames frames.
wavernn_status launch_cond(const wavernn_model* m, const float* feat, int64_t n_frames, int n_streams, float* cb,
                           hipStream_t st) {
  const float* Wc = m->d_Wc;
  const float* bias = m->d_bias;
  int dc = m->cfg.cond_dim;
  int rows = 3 * m->cfg.hidden;
  int64_t nf = n_frames;
  int ns = n_streams;
  void* args[] = {&Wc, &bias, &feat, &dc, &rows, &nf, &ns, &cb};
  const int64_t n = (int64_t)n_streams * n_frames * rows;
  HIPOK(hipLaunchKernel(wr_cond_kernel_ptr(), dim3((unsigned)((n + 255) / 256)), dim3(256), args, 0, st));
  return WAVERNN_OK;
}

// Zero n exchange words (as (n + 1) / 2 64-bit stores; buffers are sized for that).
wavernn_status launch_fill(xw* words, int64_t n_words, hipStream_t st) {
  u64* p = (u64*)words;
  int64_t n = (n_words + 1) / 2;
  int64_t nb = (n + 255) / 256;
  u64 zero = 0;
  void* args[] = {&p, &n, &zero};
  HIPOK(hipLaunchKernel(wr_fill_kernel_ptr(), dim3((unsigned)nb), dim3(256), args, 0, st));
  return WAVERNN_OK;
}

struct RunIO {
  int32_t S;
  int64_t T;
  const float* cond;
  int64_t n_frames;
  uint64_t seed;
  const wavernn_state* init;
  const wavernn_state* fin;
  const uint16_t* target;
  uint16_t* out;
  float* zc;
  float* zf;
  float* nll;
  hipStream_t st;
  unsigned char* ws = nullptr;   // caller-provided workspace (device) instead of the model's buffers, or null
  size_t ws_cap = 0;             // its bytes
  int64_t step0 = 0;             // subscale: the schedule steps [step0, step0 + n_steps) of the call run
  int64_t n_steps = -1;          // (-1: the whole schedule, a wavernn_sample call)
};

inline size_t rup256(size_t n) { return (n + 255) / 256 * 256; }

// Exchange words and a per-frame table for each of n_launch launches, carved
// from the call's workspace: [launch][exchange words | table], 256-byte aligned.
wavernn_status carve_ws(const RunIO& io, int n_launch, size_t x_words, size_t cb_floats, xw** xc, float** cb) {
  const size_t xb = rup256((x_words + 1) / 2 * 8), cbb = rup256(cb_floats * 4), per = xb + cbb;
  if (per * (size_t)n_launch > io.ws_cap)
    return fail(WAVERNN_E_INVALID, "the call needs %zu bytes of workspace (%d launch(es) x (%zu exchange + %zu table)), "
                "more than the %zu available", per * (size_t)n_launch, n_launch, xb, cbb, io.ws_cap);
  for (int i = 0; i < n_launch; ++i) {
    xc[i] = (xw*)(io.ws + per * i);
    cb[i] = (float*)(io.ws + per * i + xb);
  }
  return WAVERNN_OK;
}

wavernn_status validate_run(wavernn_model* m, const RunIO& io) {
  if (!m) return fail(WAVERNN_E_INVALID, "null model");
  const wavernn_config& c = m->cfg;
  if (io.S < 1 || io.S > c.max_streams) return fail(WAVERNN_E_INVALID, "n_streams %d not in [1, %d]", io.S, c.max_streams);
  if (io.T < 0) return fail(WAVERNN_E_INVALID, "negative n_samples");
  if (io.T > ((int64_t)1 << 31)) return fail(WAVERNN_E_INVALID, "n_samples above 2^31");
  if (c.subscale > 1 && io.T % c.subscale) return fail(WAVERNN_E_INVALID, "n_samples not a multiple of subscale");
  const int64_t t0 = io.init ? io.init->t0 : 0;
  if (t0 < 0) return fail(WAVERNN_E_INVALID, "negative t0");
  if (c.subscale > 1 && t0 != 0) return fail(WAVERNN_E_INVALID, "t0 must be 0 with subscale");
  if (c.fused && io.T > ((int64_t)1 << 30)) return fail(WAVERNN_E_INVALID, "n_samples above 2^30 for a fused model");
  if (io.init && (!io.init->h || !io.init->c_prev || !io.init->f_prev))
    return fail(WAVERNN_E_INVALID, "init state has a null pointer");
  if (io.fin && (!io.fin->h || !io.fin->c_prev || !io.fin->f_prev))
    return fail(WAVERNN_E_INVALID, "final state has a null pointer");
  if (c.cond_dim > 0) {
    if (!io.cond) return fail(WAVERNN_E_INVALID, "cond is null with cond_dim > 0");
    int64_t need = io.T > 0 ? (t0 + io.T - 1) / c.frame_len + 1 : 0;
    if (io.n_frames < need) return fail(WAVERNN_E_INVALID, "n_frames %lld < %lld frames needed", (long long)io.n_frames, (long long)need);
  }
  if (io.T > 0 && !io.target && !io.out) return fail(WAVERNN_E_INVALID, "out is null");
  return WAVERNN_OK;
}

wavernn_status run_small(wavernn_model* m, const RunIO& io) {
  SmallArgs a;
  memset(&a, 0, sizeof a);
  a.image = m->d_image;
  a.Wc = m->d_Wc;
  a.feat = io.cond;
  a.n_frames = io.n_frames;
  a.H = m->cfg.hidden;
  a.Dc = m->cfg.cond_dim;
  a.frame_len = m->cfg.frame_len > 0 ? m->cfg.frame_len : 1;
  a.T = io.T;
  a.t0 = io.init ? io.init->t0 : 0;
  a.seed = io.seed;
  a.target = io.target;
  a.out = io.out;
  a.zc_out = io.zc;
  a.zf_out = io.zf;
  a.nll_out = io.nll;
  if (io.init) { a.h_in = io.init->h; a.c_in = io.init->c_prev; a.f_in = io.init->f_prev; }
  if (io.fin) { a.h_out = io.fin->h; a.c_out = io.fin->c_prev; a.f_out = io.fin->f_prev; }
  void* args[] = {&a};
  HIPOK(hipLaunchKernel(wr_small_kernel_ptr(), dim3(io.S), dim3(256), args, m->sl.total_floats * 4, io.st));
  return WAVERNN_OK;
}

// One persistent launch for utterance s of the call, with exchange words xc
// and bias + conditioning table cb, on stream st.  A launch that runs alone
// (fan = 0) takes the tuned placement, one of fan side by side the placement
// of fan_plan.
PersistPlan solo_plan(const wavernn_model* m) {
  PersistPlan P = m->plan;
  wr_place(&P, m->solo_hx, m->solo_uxm);
  return P;
}

wavernn_status launch_persist_one(wavernn_model* m, const RunIO& io, int s, xw* xc, float* cb, int64_t n_cb,
                                  hipStream_t st, int fan) {
  const PersistPlan P = fan ? fan_plan(m, s, fan) : solo_plan(m);
  const int H = P.H, Dc = m->cfg.cond_dim;
  const int frame_len = m->cfg.frame_len > 0 ? m->cfg.frame_len : 1;
  {
    const float* feat = io.cond ? io.cond + (size_t)s * io.n_frames * Dc : nullptr;
    wavernn_status c = launch_cond(m, feat, n_cb, 1, cb, st);
    if (c != WAVERNN_OK) return c;
  }
  wavernn_status stt = launch_fill(xc, P.x_words, st);
  if (stt != WAVERNN_OK) return stt;
  PersistArgs a;
  memset(&a, 0, sizeof a);
  a.P = P;
  a.hw = m->d_hw;
  a.uw = m->d_uw;
  a.ur = m->d_ur;
  a.mw = m->d_mw;
  a.Iw = m->d_I;
  a.b1 = m->d_b1;
  a.b2 = m->d_b2;
  a.b3 = m->d_b3;
  a.b4 = m->d_b4;
  a.cb = cb;
  a.n_cb = n_cb;
  a.frame_len = Dc > 0 ? frame_len : (1 << 30);
  // fused 2x: N / 2 positions per sub-tensor, sub-tensor 1 F + 1 steps behind;
  // 32 logits per sample and byte; two last samples per utterance
  const int nz = m->fused ? 32 : 256, nb = m->fused ? 2 : 1;
  a.F = m->fused ? m->cfg.future_horizon : 0;
  a.rows = m->fused ? io.T / 2 : io.T;
  a.T = m->fused ? a.rows + a.F + 1 : io.T;
  a.t0 = io.init ? io.init->t0 : 0;
  a.seed = io.seed;
  a.stream_id = (uint64_t)s;
  a.target = io.target ? io.target + (size_t)s * io.T : nullptr;
  a.out = io.out ? io.out + (size_t)s * io.T : nullptr;
  a.zc_out = io.zc ? io.zc + (size_t)s * io.T * nz : nullptr;
  a.zf_out = io.zf ? io.zf + (size_t)s * io.T * nz : nullptr;
  a.nll_out = io.nll ? io.nll + (size_t)s * io.T : nullptr;
  if (io.init) {
    a.h_in = io.init->h + (size_t)s * H;
    a.c_in = io.init->c_prev + (size_t)nb * s;
    a.f_in = io.init->f_prev + (size_t)nb * s;
  }
  if (io.fin) {
    a.h_out = io.fin->h + (size_t)s * H;
    a.c_out = io.fin->c_prev + (size_t)nb * s;
    a.f_out = io.fin->f_prev + (size_t)nb * s;
  }
  a.xc = xc;
  a.err = m->d_err;
  a.limit = kWaitTicks;
  if (s == 0) {
    a.trace = m->trace;
    a.trace_steps = m->trace ? m->trace_steps : 0;
  }
  void* args[] = {&a};
  // An ordinary launch: create() checked that the whole grid fits on the
  // device at once, and every cross-workgroup wait is bounded, so a grid
  // that did not become co-resident ends with an error, never a hang.
  HIPOK(hipLaunchKernel(m->pk, dim3(P.grid), dim3(WR_THREADS), args, P.lds, st));
  return WAVERNN_OK;
}

// Grow a per-frame table to n_cb frames (the only allocation a call can
// make; a replaced table stays allocated until the model is destroyed, so a
// launch still reading it is unaffected).
wavernn_status grow_cb(wavernn_model* m, float** cb, int64_t* cap, int64_t n_cb) {
  if (n_cb <= *cap) return WAVERNN_OK;
  float* p = nullptr;
  wavernn_status s = m->alloc(&p, (size_t)n_cb * 3 * m->plan.H * 4);
  if (s != WAVERNN_OK) return s;
  *cb = p;
  *cap = n_cb;
  return WAVERNN_OK;
}

// Several utterances one after another on the caller's stream.
wavernn_status run_persist(wavernn_model* m, const RunIO& io) {
  const int64_t n_cb = m->cfg.cond_dim > 0 ? io.n_frames : 1;
  if (io.ws) {   // every launch of the call reuses one region of the workspace, in stream order
    xw* xc;
    float* cb;
    wavernn_status st = carve_ws(io, 1, m->plan.x_words, (size_t)n_cb * 3 * m->plan.H, &xc, &cb);
    for (int s = 0; s < io.S && st == WAVERNN_OK; ++s) st = launch_persist_one(m, io, s, xc, cb, n_cb, io.st, 0);
    return st;
  }
  if (n_cb > m->cb_cap) HIPOK(hipStreamSynchronize(io.st));
  wavernn_status st = grow_cb(m, &m->d_cb, &m->cb_cap, n_cb);
  if (st != WAVERNN_OK) return st;
  for (int s = 0; s < io.S; ++s)
    if ((st = launch_persist_one(m, io, s, m->d_xc, m->d_cb, n_cb, io.st, 0)) != WAVERNN_OK) return st;
  return WAVERNN_OK;
}

// Teacher-forced scoring of one or more utterances on the dense batch-1 plan
// (Sec. 5's NLL; Eq. 2 with the bytes given).  Per utterance the scoring
// kernel runs the recurrence and writes h after every step; then the output
// layers of all steps run as GEMMs on the matrix cores (O2 relu(O1 y_c + b1)
// + b2, the same for the fine half; up to 65,536 steps at a time) and the
// NLL as one reduction per step.
wavernn_status run_score(wavernn_model* m, const RunIO& io) {
  const int Hh = m->plan.Hh, NP = m->sc_np;
  const int64_t rows = (int64_t)io.S * io.T, CH = 65536;
  const int64_t n_cb = m->cfg.cond_dim > 0 ? io.n_frames : 1;
  const bool post = io.zc || io.zf || io.nll;
  const int64_t ch = std::min(CH, rows);   // rows of one chunk of the output layers
  // Up to nfan utterances: one single-utterance grid each, side by side on
  // the caller's stream and the internal ones (measured faster than one grid
  // carrying them); more: launches of up to 8 on the several-utterance
  // kernel, nfan of them side by side.  Each slot has its own exchange words
  // and table; all are joined before the output layers.
  const int nf = m->score_fan ? m->nfan : 1;
  const int LV = io.S > nf && m->smk ? 8 : 1;
  const int G = (io.S + LV - 1) / LV;
  const int conc = std::min(G, nf);
  const bool slots = conc > 1 || LV > 1;   // per-slot buffers (else the model's own)
  const int H = m->plan.H, Dc = m->cfg.cond_dim;
  const int64_t cbf = (int64_t)8 * n_cb * 3 * H;    // table floats per slot (up to 8 utterances)
  if (rows > m->traj_cap || (post && ch > m->so_cap) || n_cb > m->cb_cap || (slots && cbf > m->scb_cap))
    HIPOK(hipStreamSynchronize(io.st));
  wavernn_status st = grow_cb(m, &m->d_cb, &m->cb_cap, n_cb);
  if (st != WAVERNN_OK) return st;
  if (slots) {
    for (int i = 0; i < WR_FAN; ++i)
      if (!m->d_sxc[i] && (st = m->alloc(&m->d_sxc[i], (size_t)(2 * 8 * H + 1) / 2 * 8)) != WAVERNN_OK) return st;
    if (cbf > m->scb_cap) {
      for (int i = 0; i < WR_FAN; ++i)
        if ((st = m->alloc(&m->d_scb[i], (size_t)cbf * 4)) != WAVERNN_OK) return st;
      m->scb_cap = cbf;
    }
  }
  if (rows > m->traj_cap) {
    if ((st = m->alloc(&m->d_traj, (size_t)2 * rows * Hh * 4)) != WAVERNN_OK) return st;
    m->traj_cap = rows;
  }
  if (post && ch > m->so_cap) {   // (a replaced buffer stays allocated until the model is destroyed)
    if ((st = m->alloc(&m->d_so, (size_t)ch * NP * 4)) != WAVERNN_OK) return st;
    if ((st = m->alloc(&m->d_sz, (size_t)2 * ch * 256 * 4)) != WAVERNN_OK) return st;
    m->so_cap = ch;
  }
  if (conc > 1) HIPOK(hipEventRecord(m->fan_fork, io.st));
  for (int g = 0; g < G; ++g) {
    const int slot = g % conc, s0 = g * LV, nv = std::min(LV, io.S - s0);
    hipStream_t sst = slot > 0 ? m->fan_st[slot - 1] : io.st;
    xw* xc = slots ? m->d_sxc[slot] : m->d_xc;
    float* cbt = slots ? m->d_scb[slot] : m->d_cb;
    if (slot > 0 && g < conc) HIPOK(hipStreamWaitEvent(sst, m->fan_fork, 0));
    const float* feat = io.cond ? io.cond + (size_t)s0 * io.n_frames * Dc : nullptr;
    if ((st = launch_cond(m, feat, n_cb, nv, cbt, sst)) != WAVERNN_OK) return st;
    if ((st = launch_fill(xc, 2 * LV * H, sst)) != WAVERNN_OK) return st;
    ScoreArgs a;
    memset(&a, 0, sizeof a);
    a.w = m->d_srw;
    a.Iw = m->d_I;
    a.cb = cbt;
    a.n_cb = n_cb;
    a.frame_len = Dc > 0 ? (m->cfg.frame_len > 0 ? m->cfg.frame_len : 1) : (1 << 30);
    a.H = H;
    a.Hh = Hh;
    a.T = io.T;
    a.t0 = io.init ? io.init->t0 : 0;
    a.target = io.target + (size_t)s0 * io.T;
    if (io.init) {
      a.h_in = io.init->h + (size_t)s0 * H;
      a.c_in = io.init->c_prev + s0;
      a.f_in = io.init->f_prev + s0;
    }
    if (io.fin) {
      a.h_out = io.fin->h + (size_t)s0 * H;
      a.c_out = io.fin->c_prev + s0;
      a.f_out = io.fin->f_prev + s0;
    }
    a.traj_c = m->d_traj + (size_t)s0 * io.T * Hh;
    a.traj_f = m->d_traj + (size_t)(io.S + s0) * io.T * Hh;
    a.xc = xc;
    a.err = m->d_err;
    a.limit = kWaitTicks;
    a.nv = nv;
    void* args[] = {&a};
    // an ordinary launch of H / 16 workgroups (co-residency checked at create; waits bounded)
    if (LV > 1)
      HIPOK(hipLaunchKernel(m->smk, dim3(H / 16), dim3(WR_THREADS), args, score_multi_lds(H), sst));
    else
      HIPOK(hipLaunchKernel(m->sk, dim3(H / 16), dim3(WR_THREADS), args, score_lds(H), sst));
  }
  for (int i = 1; i < conc; ++i) {
    HIPOK(hipEventRecord(m->fan_join[i - 1], m->fan_st[i - 1]));
    HIPOK(hipStreamWaitEvent(io.st, m->fan_join[i - 1], 0));
  }
  if (!post) return WAVERNN_OK;
  for (int64_t r0 = 0; r0 < rows; r0 += CH) {
    const int n = (int)std::min(CH, rows - r0);
    const CnnRows cr{1, 0, 0, n};
    float* z[2];
    for (int k = 0; k < 2; ++k) {
      float* user = k ? io.zf : io.zc;
      z[k] = user ? user + (size_t)r0 * 256 : m->d_sz + (size_t)k * ch * 256;
      const float* src = m->d_traj + ((size_t)k * rows + r0) * Hh;
      if ((st = cnn_gemm(src, Hh, 1, 0, n, cr, n, m->d_sw + m->sw_off[2 * k], m->d_sb + m->sb_off[2 * k], NP,
                         m->d_so, 1, io.st)) != WAVERNN_OK)
        return st;
      if ((st = cnn_gemm(m->d_so, NP, 1, 0, n, cr, n, m->d_sw + m->sw_off[2 * k + 1], m->d_sb + m->sb_off[2 * k + 1],
                         256, z[k], 0, io.st)) != WAVERNN_OK)
        return st;
    }
    if (io.nll) {
      const float* zc = z[0];
      const float* zf = z[1];
      const uint16_t* tg = io.target + r0;
      int64_t nn = n;
      float* nl = io.nll + r0;
      void* args[] = {&zc, &zf, &tg, &nn, &nl};
      HIPOK(hipLaunchKernel(wr_score_nll_ptr(), dim3((unsigned)((n + 3) / 4)), dim3(256), args, 0, io.st));
    }
  }
  return WAVERNN_OK;
}

// A few utterances at once: utterance 0 runs the batch-1 kernel on the
// caller's stream, utterance s > 0 on internal stream s - 1 (each its own
// grid, exchange words and table), forked from and joined back into the
// caller's stream, so the call stays stream-ordered.  The grids are
// co-resident together (checked at create); with one hardware queue per
// stream (4 by default, so the caller's stream and 3 more) the launches run
// side by side: at batch 4 about four times the batch-1 rate, where the
// batched kernel, which shares one grid among the utterances, gives under
// three.
wavernn_status run_fanout(wavernn_model* m, const RunIO& io) {
  const int64_t n_cb = m->cfg.cond_dim > 0 ? io.n_frames : 1;
  wavernn_status st = WAVERNN_OK;
  xw* xc[WR_FAN] = {};
  float* cb[WR_FAN] = {};
  if (io.ws) {
    if ((st = carve_ws(io, io.S, m->plan.x_words, (size_t)n_cb * 3 * m->plan.H, xc, cb)) != WAVERNN_OK) return st;
  } else {
    for (int i = 0; i < io.S; ++i) xc[i] = m->d_fxc[i];
  }
  if (!io.ws && n_cb > m->fcb_cap) {
    HIPOK(hipStreamSynchronize(io.st));
    int64_t cap = 0;
    for (int i = 0; i < m->nfan && st == WAVERNN_OK; ++i) {
      cap = m->fcb_cap;
      st = grow_cb(m, &m->d_fcb[i], &cap, n_cb);
    }
    if (st != WAVERNN_OK) return st;
    m->fcb_cap = cap;
  }
  if (!io.ws)
    for (int i = 0; i < io.S; ++i) cb[i] = m->d_fcb[i];
  HIPOK(hipEventRecord(m->fan_fork, io.st));
  for (int s = 1; s < io.S; ++s) {
    HIPOK(hipStreamWaitEvent(m->fan_st[s - 1], m->fan_fork, 0));
    if ((st = launch_persist_one(m, io, s, xc[s], cb[s], n_cb, m->fan_st[s - 1], io.S)) != WAVERNN_OK) return st;
    HIPOK(hipEventRecord(m->fan_join[s - 1], m->fan_st[s - 1]));
  }
  if ((st = launch_persist_one(m, io, 0, xc[0], cb[0], n_cb, io.st, io.S)) != WAVERNN_OK) return st;
  for (int s = 1; s < io.S; ++s) HIPOK(hipStreamWaitEvent(io.st, m->fan_join[s - 1], 0));
  return WAVERNN_OK;
}

wavernn_status run_batch(wavernn_model* m, const RunIO& io) {
  const int SB = m->cfg.subscale;                 // lanes per utterance
  const int V = io.S * SB;                        // vectors
  BatchPlan B;
  const int F = horizon_of(m->cfg), A = lead_of(m->cfg);
  const bool table = m->has_cnn;
  if (!batch_plan(m->cfg.hidden, V, &B, m->cfg.ctx_dim, SB, F, A, table))
    return fail(WAVERNN_E_UNSUPPORTED, "no batched plan for %d vectors", V);
  if (table && io.ws) return fail(WAVERNN_E_UNSUPPORTED, "the conditioning CNN needs its own activation buffers");
  if (table && m->trace)
    return fail(WAVERNN_E_UNSUPPORTED, "phase tracing is switched off for CNN-conditioned calls (a traced call had a "
                "bounded wait expire and the cause is not found; untraced calls are unaffected)");
  const int H = B.H, Dc = m->cfg.cond_dim;
  const int frame_len = m->cfg.frame_len > 0 ? m->cfg.frame_len : 1;
  const int64_t n_cb = Dc > 0 ? io.n_frames : 1;
  const size_t need = (size_t)io.S * n_cb * 3 * H;
  xw* xc = m->d_bxc;
  float* cbt = m->d_bcb;
  wavernn_status st;
  if (io.ws) {
    if ((st = carve_ws(io, 1, (size_t)B.G * B.x_words, need, &xc, &cbt)) != WAVERNN_OK) return st;
  } else if (need > m->bcb_cap) {   // grow the per-frame table (the only allocation a call can make)
    HIPOK(hipStreamSynchronize(io.st));
    float* p = nullptr;
    wavernn_status s = m->alloc(&p, need * 4);
    if (s != WAVERNN_OK) return s;
    m->d_bcb = cbt = p;
    m->bcb_cap = need;
  }
  const void* kernel = wr_batch_kernel_ptr(B.KH, B.KX > 0, B.L, F >= 0);
  if (!kernel) return fail(WAVERNN_E_UNSUPPORTED, "no batched kernel for %d vectors", V);
  if ((st = launch_cond(m, io.cond, n_cb, io.S, cbt, io.st)) != WAVERNN_OK) return st;
  BatchArgs a;
  memset(&a, 0, sizeof a);
  a.P = B;
  a.hw = m->d_hw;
  a.uw = m->d_buw;
  a.ur = m->d_bur;
  a.Iw = m->d_I;
  a.b1 = m->d_b1;
  a.b2 = m->d_b2;
  a.b3 = m->d_b3;
  a.b4 = m->d_b4;
  a.ux = m->d_bux;
  a.cb = cbt;
  a.n_cb = n_cb;
  a.frame_len = Dc > 0 ? frame_len : (1 << 30);
  a.S = V;
  a.B = SB;
  a.F = F;
  a.A = A;
  a.rows = io.T / SB;
  a.seed = io.seed;
  a.target = io.target;
  a.out = io.out;
  a.zc_out = io.zc;
  a.zf_out = io.zf;
  a.nll_out = io.nll;
  a.xc = xc;
  a.err = m->d_err;
  a.limit = kWaitTicks;
  a.trace = m->trace;
  a.trace_steps = m->trace ? m->trace_steps : 0;
  const int64_t steps = a.rows + (F >= 0 ? (int64_t)(SB - 1) * (F + 1 + A) : 0);   // the last lane starts late
  // the steps this call runs (a resumed subscale call: a part of the schedule)
  const int64_t s0 = io.n_steps >= 0 ? io.step0 : 0, s1 = io.n_steps >= 0 ? io.step0 + io.n_steps : steps;
  // one launch of steps [t0, t0 + n) from state `in` to state `out` (null: default / nowhere)
  auto launch = [&](int64_t t0, int64_t n, const wavernn_state* in, const wavernn_state* out) -> wavernn_status {
    wavernn_status e = launch_fill(xc, (int64_t)B.G * B.x_words, io.st);
    if (e != WAVERNN_OK) return e;
    a.t0 = t0;
    a.T = n;
    if (SB > 1 && F < 0 && io.out) a.out = io.out + (size_t)SB * t0;   // lockstep rows: from row t0 on
    // a resumed window-context launch starts the units' sample rings from the utterances' buffer
    a.prev = m->cfg.ctx_dim > 0 && !table && SB > 1 && t0 > 0 ? io.out : nullptr;
    a.h_in = in ? in->h : nullptr;
    a.c_in = in ? in->c_prev : nullptr;
    a.f_in = in ? in->f_prev : nullptr;
    a.h_out = out ? out->h : nullptr;
    a.c_out = out ? out->c_prev : nullptr;
    a.f_out = out ? out->f_prev : nullptr;
    void* args[] = {&a};
    // an ordinary launch, as for the batch-1 kernel (co-residency checked at create)
    HIPOK(hipLaunchKernel(kernel, dim3(B.grid), dim3(WR_THREADS), args, B.lds, io.st));
    return WAVERNN_OK;
  };
  if (!table) return SB > 1 ? launch(s0, s1 - s0, io.init, io.fin) : launch(io.init ? io.init->t0 : 0, steps, io.init, io.fin);
  // Conditioning CNN (Sec. 4.1).  Teacher forcing: the whole context table
  // from the targets, one launch.
  const int64_t rows = a.rows;
  if (io.target) {
    hipStream_t s0 = io.st;
    if ((st = grow_ctab(m, (size_t)V * rows * m->cfg.ctx_dim, &s0)) != WAVERNN_OK) return st;
    if ((st = run_cnn(m, io.S, io.target, io.T, (int)rows, 0, 0, rows, 0, m->d_ctab, io.st)) != WAVERNN_OK) return st;
    a.ctab = m->d_ctab;
    a.ctab_rows = rows;
    a.ctab_row0 = 0;
    a.ctab_step = 0;
    return launch(0, steps, io.init, io.fin);   // (scoring runs whole calls only)
  }
  // Sampling: chunks of LC = F - R + 1 steps (R the CNN's reach in rows).
  // Before chunk [t0, t0 + LC) sub-tensor z < s has made its rows up to
  // t0 - 1 - z (F + 1), which covers the next LC rows of sub-tensor s (from its
  // position t0 - s (F + 1)) with their reach (Sec. 4.2: the conditioning runs
  // ahead by a chosen number of samples; the lag between sub-tensors pays for
  // it).  The CNN is streamed (run_cnn_stream): each chunk computes the rows
  // of every layer that have become final, into a whole-utterance table.  The
  // call's first chunk starts every level at the first position the call runs.
  if (SB > WR_CNN_MAXB || m->cnn.layers + 2 > 2 * 32 + 2)
    return fail(WAVERNN_E_UNSUPPORTED, "streamed CNN: at most %d sub-tensors and 64 layers", WR_CNN_MAXB);
  const int64_t LC = m->cnn_chunk;
  {
    hipStream_t s0s = io.st;
    if ((st = grow_ctab(m, (size_t)V * rows * m->cfg.ctx_dim, &s0s)) != WAVERNN_OK) return st;
  }
  a.ctab = m->d_ctab;
  a.ctab_rows = rows;
  a.ctab_row0 = 0;
  a.ctab_step = 0;
  int lo[2 * 32 + 2][WR_CNN_MAXB];
  for (int v = 0; v < m->cnn.layers + 2; ++v)
    for (int s = 0; s < WR_CNN_MAXB; ++s) {
      const int64_t p = s0 - (int64_t)s * (F + 1);
      lo[v][s] = (int)(s < SB ? std::min<int64_t>(std::max<int64_t>(p, 0), rows) : 0);
    }
  int cur = 0;
  for (int64_t t0 = s0; t0 < s1; t0 += LC) {
    const int64_t n = std::min(LC, s1 - t0);
    if ((st = run_cnn_stream(m, io.S, io.out, io.T, t0, F, lo, m->d_ctab, io.st)) != WAVERNN_OK) return st;
    const bool last = t0 + n >= s1;
    const wavernn_state* in = t0 == s0 ? io.init : &m->cnn_state[cur];
    const wavernn_state* out = last ? io.fin : &m->cnn_state[cur ^ 1];
    if ((st = launch(t0, n, in, out)) != WAVERNN_OK) return st;
    cur ^= 1;
  }
  return WAVERNN_OK;
}

wavernn_status scratch_of(int dev, unsigned char** out, size_t* cap);

wavernn_status run(wavernn_model* m, RunIO& io, bool noalloc = false) {
  wavernn_status s = validate_run(m, io);
  if (s != WAVERNN_OK) return s;
  if (io.T == 0) return WAVERNN_OK;
  int dev = 0;
  HIPOK(hipGetDevice(&dev));
  if (dev != m->device) return fail(WAVERNN_E_INVALID, "model lives on device %d, current device is %d", m->device, dev);
  if (noalloc && (s = scratch_of(dev, &io.ws, &io.ws_cap)) != WAVERNN_OK) return s;
  if (m->path == PATH_SMALL) return run_small(m, io);
  if (m->fused) return run_persist(m, io);   // one fused launch per utterance
  if (m->path == PATH_PERSIST) {
    // one utterance (or a model that runs its utterances one after another) scores on the recurrence kernel
    if (io.target && m->sk && (io.S == 1 || m->smk || (io.S <= m->nfan && m->score_fan) || (!m->nfan && !m->has_batch)))
      return run_score(m, io);
    if (io.S > 1 && io.S <= m->nfan) return run_fanout(m, io);
    return io.S > 1 && m->has_batch ? run_batch(m, io) : run_persist(m, io);
  }
  if (m->path == PATH_BATCHED) return run_batch(m, io);
  return fail(WAVERNN_E_UNSUPPORTED, "no kernel for this configuration");
}

}  // namespace

// Workspace of wavernn_sample_noalloc: one array per device (each device that
// runs the library holds its own copy until the process ends).  Host code
// never uses the array's name as an address: the device address is looked up
// once per device with hipGetSymbolAddress and kept in g_scratch.
#define WR_SCRATCH_BYTES ((size_t)16 << 20)
#define WR_MAX_DEVICES 64
static __device__ __align__(256) uint64_t scratch[WR_SCRATCH_BYTES / 8];

namespace {

std::mutex g_scratch_mu;
unsigned char* g_scratch[WR_MAX_DEVICES] = {};

// Device address of the workspace on device `dev`, which must be current.
wavernn_status scratch_of(int dev, unsigned char** out, size_t* cap) {
  if (dev < 0 || dev >= WR_MAX_DEVICES) return fail(WAVERNN_E_UNSUPPORTED, "device %d: above %d devices", dev, WR_MAX_DEVICES);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(WAVERNN_E_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch[dev] = (unsigned char*)p;
  }
  *out = g_scratch[dev];
  *cap = WR_SCRATCH_BYTES;
  return WAVERNN_OK;
}

// Mean microseconds per step of one launch of `k` (HIP events on `st`).
wavernn_status time_launch(wavernn_model* m, const void* k, int grid, int lds, void* arg, int64_t steps, double* us,
                           hipStream_t st) {
  void* args[] = {arg};
  hipEvent_t e0, e1;
  HIPOK(hipEventCreate(&e0));
  HIPOK(hipEventCreate(&e1));
  hipError_t he = hipEventRecord(e0, st);
  if (he == hipSuccess) he = hipLaunchKernel(k, dim3(grid), dim3(WR_THREADS), args, lds, st);
  if (he == hipSuccess) he = hipEventRecord(e1, st);
  if (he == hipSuccess) he = hipEventSynchronize(e1);
  float ms = 0.0f;
  if (he == hipSuccess) he = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (he != hipSuccess) return fail(WAVERNN_E_HIP, "sync floor: %s", hipGetErrorString(he));
  *us = (double)ms * 1000.0 / (double)steps;
  return wavernn_device_status(m, st);
}

// The floor of the batched launch a call on max_streams utterances makes:
// the batched kernel itself with its arithmetic compiled out (same plan,
// grid, roles, exchanged words, class and sample words, waits and barriers).
wavernn_status batch_floor(wavernn_model* m, int64_t n_steps, double* us, hipStream_t st) {
  const int SB = m->cfg.subscale, V = m->cfg.max_streams * SB;
  const int F = horizon_of(m->cfg), A = lead_of(m->cfg);
  if (m->has_cnn) return fail(WAVERNN_E_UNSUPPORTED, "no sync floor for a model with a conditioning CNN");
  BatchPlan B;
  if (!batch_plan(m->cfg.hidden, V, &B, m->cfg.ctx_dim, SB, F, A))
    return fail(WAVERNN_E_UNSUPPORTED, "no batched plan for %d vectors", V);
  const void* k = wr_batch_floor_kernel_ptr(B.KH, B.KX > 0, B.L, F >= 0);
  if (!k) return fail(WAVERNN_E_UNSUPPORTED, "hidden %d: no batched floor instantiation", B.H);
  wavernn_status s = check_coresident(m, k, B.grid, B.lds, "batched sync-floor");
  if (s != WAVERNN_OK) return s;
  const size_t cbn = (size_t)m->cfg.max_streams * 3 * B.H;   // one frame of bias + conditioning (zeros)
  if (cbn > m->bcb_cap) {
    float* p = nullptr;
    if ((s = m->alloc(&p, cbn * 4)) != WAVERNN_OK) return s;
    m->d_bcb = p;
    m->bcb_cap = cbn;
  }
  if ((s = launch_fill((xw*)m->d_bcb, (int64_t)cbn, st)) != WAVERNN_OK) return s;
  if ((s = launch_fill(m->d_bxc, (int64_t)B.G * B.x_words, st)) != WAVERNN_OK) return s;
  BatchArgs a;
  memset(&a, 0, sizeof a);
  a.P = B;
  a.hw = m->d_hw;
  a.uw = m->d_buw;
  a.ur = m->d_bur;
  a.Iw = m->d_I;
  a.b1 = m->d_b1;
  a.b2 = m->d_b2;
  a.b3 = m->d_b3;
  a.b4 = m->d_b4;
  a.ux = m->d_bux;
  a.cb = m->d_bcb;
  a.n_cb = 1;
  a.frame_len = 1 << 30;
  a.S = V;
  a.B = SB;
  a.F = F;
  a.A = A;
  a.rows = n_steps;
  a.T = n_steps + (F >= 0 ? (int64_t)(SB - 1) * (F + 1 + A) : 0);
  a.xc = m->d_bxc;
  a.err = m->d_err;
  a.limit = kWaitTicks;
  return time_launch(m, k, B.grid, B.lds, &a, a.T, us, st);
}

}  // namespace

extern "C" {

wavernn_status wavernn_create(const wavernn_config* cfg, const wavernn_weights* w, wavernn_model** out) {
  if (!out) return fail(WAVERNN_E_INVALID, "null output handle");
  *out = nullptr;
  wavernn_status s = validate_config(cfg, w);
  if (s != WAVERNN_OK) return s;
  wavernn_model* m = new (std::nothrow) wavernn_model();
  if (!m) return fail(WAVERNN_E_OOM, "host allocation failed");
  m->cfg = *cfg;
  if (hipGetDevice(&m->device) != hipSuccess) {
    delete m;
    return fail(WAVERNN_E_HIP, "no HIP device");
  }
  const int H = cfg->hidden;
  const SmallLayout L = small_layout(H);
  const bool small_fits = (size_t)L.total_floats * 4 + 256 <= 160 * 1024;
  const int B = cfg->subscale;
  if (cfg->fused) {
    // Fused Subscale WaveRNN 2x (Sec. 4.4): the batch-1 persistent structure
    // with fused heads, one launch per utterance
    if (cfg->weight_dtype != WAVERNN_BF16)
      s = fail(WAVERNN_E_UNSUPPORTED, "fused 2x sampling needs bf16 weights");
    else if (!fused_plan(H, &m->plan))
      s = fail(WAVERNN_E_UNSUPPORTED, "hidden %d: no fused plan (need a multiple of 128 up to 896)", H);
    else {
      m->path = PATH_PERSIST;
      s = build_fused(m, w);
    }
  } else if (B > 1) {
    // Subscale (Sec. 4): the B lanes of each utterance are vectors of the
    // batched kernel; its unit workgroups add the context projection.
    if (!((B % 8 == 0) || (4 % B == 0)) || cfg->ctx_dim % 32 || cfg->ctx_dim > 256)
      s = fail(WAVERNN_E_UNSUPPORTED, "subscale %d / ctx_dim %d: need B a multiple of 8 or a divisor of 4 (lanes "
               "must tile groups of 2, 4 and 8 vectors), ctx_dim a multiple of 32 up to 256", B, cfg->ctx_dim);
    else if (cfg->weight_dtype != WAVERNN_BF16)
      s = fail(WAVERNN_E_UNSUPPORTED, "subscale sampling needs bf16 weights");
    else if ((m->has_cnn = w->ctx_cnn != nullptr) && cnn_reach(w->ctx_cnn->layers) > cfg->future_horizon)
      s = fail(WAVERNN_E_INVALID, "ctx_cnn: the future horizon %d is below the CNN's reach of %d rows (the "
               "CNN runs ahead in chunks of F - reach + 1 steps)", cfg->future_horizon, cnn_reach(w->ctx_cnn->layers));
    else if (!persist_plan(H, &m->plan) ||
             !batch_plan(H, cfg->max_streams * B, &m->bplan, cfg->ctx_dim, B, horizon_of(*cfg), lead_of(*cfg),
                         m->has_cnn))
      s = fail(WAVERNN_E_UNSUPPORTED, "hidden %d with %d x %d lanes, future horizon %d, context lead %d: no batched "
               "plan (the units' ring of B (B - 1)(F + 1 + A) + Dx/2 + B samples must fit LDS)", H, cfg->max_streams,
               B, horizon_of(*cfg), lead_of(*cfg));
    else {
      m->path = PATH_BATCHED;
      s = build_persist(m, w);
      if (s == WAVERNN_OK) s = build_batch(m, w);
      if (s == WAVERNN_OK && w->ctx_cnn) s = build_cnn(m, w->ctx_cnn);
      if (s == WAVERNN_OK && w->ctx_cnn) {   // sampling chunks, their context window and the state between them
        const int R = cnn_reach(w->ctx_cnn->layers), V = cfg->max_streams * B;
        m->cnn_chunk = cfg->future_horizon - R + 1;
        m->cnn_win = m->cnn_chunk + R;
        s = grow_ctab(m, (size_t)V * m->cnn_win * cfg->ctx_dim, nullptr);
        for (int i = 0; i < 2 && s == WAVERNN_OK; ++i) {
          s = m->alloc(&m->cnn_state[i].h, (size_t)V * H * 4);
          if (s == WAVERNN_OK) s = m->alloc(&m->cnn_state[i].c_prev, V);
          if (s == WAVERNN_OK) s = m->alloc(&m->cnn_state[i].f_prev, V);
        }
      }
    }
  } else if (small_fits) {
    m->path = PATH_SMALL;
    s = build_small(m, w);
  } else if (cfg->r_format != WAVERNN_R_DENSE) {
    // Sparse WaveRNN (Sec. 3): block-sparse unit workgroups; several streams
    // run one after another
    if (cfg->weight_dtype != WAVERNN_BF16) {
      s = fail(WAVERNN_E_UNSUPPORTED, "hidden %d needs bf16 weights (fp32 weights fit LDS only for small models)", H);
    } else {
      m->path = PATH_PERSIST;
      s = build_sparse(m, w);
    }
  } else if (persist_plan(H, &m->plan)) {
    if (cfg->weight_dtype != WAVERNN_BF16) {
      s = fail(WAVERNN_E_UNSUPPORTED, "hidden %d needs bf16 weights (fp32 weights fit LDS only for small models)", H);
    } else {
      m->path = PATH_PERSIST;
      s = build_persist(m, w);
      if (s == WAVERNN_OK) s = build_score(m, w);
      if (s == WAVERNN_OK && cfg->max_streams > 1 && batch_plan(H, cfg->max_streams, &m->bplan))
        s = build_batch(m, w);
      if (s == WAVERNN_OK && cfg->max_streams > 1) s = build_fanout(m);
    }
  } else {
    s = fail(WAVERNN_E_UNSUPPORTED, "hidden %d: no kernel plan (need a multiple of 128 whose blocks fit LDS)", H);
  }
  if (s == WAVERNN_OK) {
    s = m->alloc(&m->d_err, 64);
    if (s == WAVERNN_OK && hipMemset(m->d_err, 0, 64) != hipSuccess) s = fail(WAVERNN_E_HIP, "hipMemset failed");
  }
  if (s != WAVERNN_OK) {
    delete m;
    return s;
  }
  *out = m;
  return WAVERNN_OK;
}

void wavernn_destroy(wavernn_model* m) { delete m; }

wavernn_status wavernn_sample(wavernn_model* m, int32_t n_streams, int64_t n_samples, const float* cond_dev,
                              int64_t n_frames, uint64_t seed, const wavernn_state* init, uint16_t* out_dev,
                              const wavernn_state* final_state, void* stream) {
  RunIO io{n_streams, n_samples, cond_dev, n_frames, seed, init, final_state, nullptr, out_dev,
           nullptr, nullptr, nullptr, (hipStream_t)stream};
  return run(m, io);
}

int64_t wavernn_schedule_steps(const wavernn_model* m, int64_t n_samples) {
  if (!m || m->cfg.subscale <= 1 || m->fused || m->path != PATH_BATCHED) return -1;
  const int B = m->cfg.subscale, F = horizon_of(m->cfg), A = lead_of(m->cfg);
  if (n_samples < 0 || n_samples > ((int64_t)1 << 31) || n_samples % B) return -1;
  return n_samples / B + (F >= 0 ? (int64_t)(B - 1) * (F + 1 + A) : 0);
}

wavernn_status wavernn_sample_steps(wavernn_model* m, int32_t n_streams, int64_t n_samples, const float* cond_dev,
                                    int64_t n_frames, uint64_t seed, int64_t step0, int64_t n_steps,
                                    const wavernn_state* init, uint16_t* out_dev, const wavernn_state* final_state,
                                    void* stream) {
  if (!m) return fail(WAVERNN_E_INVALID, "null model");
  if (m->cfg.subscale <= 1 || m->fused || m->path != PATH_BATCHED)
    return fail(WAVERNN_E_UNSUPPORTED, "wavernn_sample_steps serves subscale models on the batched path");
  const int64_t K = wavernn_schedule_steps(m, n_samples);
  if (K < 0) return fail(WAVERNN_E_INVALID, "n_samples %lld: not a multiple of subscale in [0, 2^31]", (long long)n_samples);
  if (step0 < 0 || n_steps < 0 || step0 > K || n_steps > K - step0)
    return fail(WAVERNN_E_INVALID, "steps [%lld, %lld) outside the call's schedule of %lld steps", (long long)step0,
                (long long)(step0 + n_steps), (long long)K);
  if (n_steps == 0) return WAVERNN_OK;
  if (step0 > 0 && !init) return fail(WAVERNN_E_INVALID, "step0 > 0 needs the state after step0 - 1 (init)");
  const int B = m->cfg.subscale;
  if (step0 > 0 && m->cfg.ctx_dim > 0 && !m->has_cnn && (B & (B - 1)))
    return fail(WAVERNN_E_UNSUPPORTED, "resuming a window-context call needs B a power of two (B = %d)", B);
  RunIO io{n_streams, n_samples, cond_dev, n_frames, seed, init, final_state, nullptr, out_dev,
           nullptr, nullptr, nullptr, (hipStream_t)stream};
  io.step0 = step0;
  io.n_steps = n_steps;
  return run(m, io);
}

wavernn_status wavernn_sample_noalloc(wavernn_model* m, int32_t n_streams, int64_t n_samples, const float* cond_dev,
                                      int64_t n_frames, uint64_t seed, const wavernn_state* init, uint16_t* out_dev,
                                      const wavernn_state* final_state, void* stream) {
  RunIO io{n_streams, n_samples, cond_dev, n_frames, seed, init, final_state, nullptr, out_dev,
           nullptr, nullptr, nullptr, (hipStream_t)stream};
  return run(m, io, true);
}

wavernn_status wavernn_score_teacher_forced(wavernn_model* m, int32_t n_streams, int64_t n_samples,
                                            const float* cond_dev, int64_t n_frames, const uint16_t* target_dev,
                                            const wavernn_state* init, float* logits_c_dev, float* logits_f_dev,
                                            float* nll_dev, void* stream) {
  if (!target_dev && n_samples != 0) return fail(WAVERNN_E_INVALID, "target is null");
  RunIO io{n_streams, n_samples, cond_dev, n_frames, 0, init, nullptr, target_dev, nullptr,
           logits_c_dev, logits_f_dev, nll_dev, (hipStream_t)stream};
  return run(m, io);
}

wavernn_status wavernn_device_status(wavernn_model* m, void* stream) {
  if (!m) return fail(WAVERNN_E_INVALID, "null model");
  HIPOK(hipStreamSynchronize((hipStream_t)stream));
  unsigned e[16];
  HIPOK(hipMemcpy(e, m->d_err, sizeof e, hipMemcpyDeviceToHost));
  if (e[0]) {
    HIPOK(hipMemset(m->d_err, 0, 64));
    return fail(WAVERNN_E_DEVICE, "kernel reported error bits 0x%x (1 = a bounded wait expired)", e[0]);
  }
  return WAVERNN_OK;
}

wavernn_status wavernn_debug_uniforms(uint64_t seed, uint64_t stream_id, int64_t t0, int64_t n, float* out_dev,
                                      void* stream) {
  if (n < 0 || (n > 0 && !out_dev) || t0 < 0) return fail(WAVERNN_E_INVALID, "bad arguments");
  if (n == 0) return WAVERNN_OK;
  void* args[] = {&seed, &stream_id, &t0, &n, &out_dev};
  HIPOK(hipLaunchKernel(wr_uniforms_kernel_ptr(), dim3((unsigned)((n + 255) / 256)), dim3(256), args, 0,
                        (hipStream_t)stream));
  return WAVERNN_OK;
}

int32_t wavernn_model_path(const wavernn_model* m, int32_t n_streams, int32_t* grid, int32_t* block) {
  if (!m) return -1;
  int g = 0, b = 0, path = (int)m->path;
  BatchPlan B;
  if (m->path == PATH_SMALL) {
    g = n_streams > 0 ? n_streams : 1, b = 256;
  } else if (m->path == PATH_BATCHED &&
             batch_plan(m->cfg.hidden, (n_streams > 0 ? n_streams : 1) * m->cfg.subscale, &B, m->cfg.ctx_dim,
                        m->cfg.subscale, horizon_of(m->cfg), lead_of(m->cfg), m->has_cnn)) {
    g = B.grid, b = WR_THREADS;
  } else if (m->path == PATH_PERSIST && n_streams > 1 && n_streams <= m->nfan) {
    path = PATH_CONCURRENT_ID, g = m->plan.grid, b = WR_THREADS;
  } else if (m->path == PATH_PERSIST && n_streams > 1 && m->has_batch && batch_plan(m->cfg.hidden, n_streams, &B)) {
    path = PATH_BATCHED, g = B.grid, b = WR_THREADS;
  } else if (m->path == PATH_PERSIST) {
    g = solo_plan(m).grid, b = WR_THREADS;
    if (m->sparse) path = PATH_SPARSE_ID;
    if (m->fused) path = PATH_FUSED_ID;
  }
  if (grid) *grid = g;
  if (block) *block = b;
  return (int32_t)path;
}

wavernn_status wavernn_debug_sync_floor(wavernn_model* m, int64_t n_steps, double* us_per_step, void* stream) {
  if (!m || n_steps < 2 || n_steps > ((int64_t)1 << 31) || !us_per_step)
    return fail(WAVERNN_E_INVALID, "bad sync-floor arguments");
  hipStream_t st = (hipStream_t)stream;
  int32_t grid = 0, block = 0;
  if (wavernn_model_path(m, m->cfg.max_streams, &grid, &block) == PATH_BATCHED) return batch_floor(m, n_steps, us_per_step, st);
  if (m->path != PATH_PERSIST) return fail(WAVERNN_E_UNSUPPORTED, "no sync floor for the single-workgroup kernel");
  if (m->fused)
    return fail(WAVERNN_E_UNSUPPORTED, "the sync floor kernel exchanges 256 partial logits per slice, not the fused "
                "heads' 64");
  const PersistPlan P = solo_plan(m);
  if ((3 * P.Hh) % P.NU) return fail(WAVERNN_E_UNSUPPORTED, "gate words do not split evenly over the units");
  const void* k = wr_floor_kernel_ptr();
  wavernn_status s = check_coresident(m, k, P.grid, P.lds, "sync-floor");
  if (s != WAVERNN_OK) return s;
  if ((s = launch_fill(m->d_xc, P.x_words, st)) != WAVERNN_OK) return s;
  PersistArgs a;
  memset(&a, 0, sizeof a);
  a.P = P;
  a.T = n_steps;
  a.xc = m->d_xc;
  a.err = m->d_err;
  a.limit = kWaitTicks;
  return time_launch(m, k, P.grid, P.lds, &a, n_steps, us_per_step, st);
}

// Placement candidate i: heads on XCD i / 8, units on XCD i % 8 (all XCDs when equal).
static void candidate_plan(const wavernn_model* m, int i, PersistPlan* P) {
  *P = m->plan;
  const int hx = i / 8, ux = i % 8;
  wr_place(P, hx, ux == hx ? 255 : 1 << ux);
}

// Does one launch of the candidate fit the device at once (every XCD holds its
// workgroups, and the grid the device)?
static wavernn_status candidate_fits(const wavernn_model* m, int i, bool* fits) {
  PersistPlan P;
  candidate_plan(m, i, &P);
  int per_cu = 0;
  HIPOK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, m->pk, WR_THREADS, P.lds));
  hipDeviceProp_t prop;
  HIPOK(hipGetDeviceProperties(&prop, m->device));
  const int per_xcd = per_cu * (prop.multiProcessorCount / 8);
  int busy[8] = {};
  for (int b = 0; b < P.grid; ++b)
    if (wr_role(P, b) >= 0) ++busy[b % 8];
  *fits = per_cu >= 1 && P.grid <= per_cu * prop.multiProcessorCount;
  for (int x = 0; x < 8; ++x) *fits = *fits && busy[x] <= per_xcd;
  return WAVERNN_OK;
}

wavernn_status wavernn_set_placement(wavernn_model* m, int32_t candidate) {
  if (!m || candidate < -1 || candidate >= 64) return fail(WAVERNN_E_INVALID, "bad placement arguments");
  if (m->path != PATH_PERSIST) return fail(WAVERNN_E_UNSUPPORTED, "the placement applies to the persistent kernels");
  if (candidate < 0) candidate = 0;
  bool fits = false;
  wavernn_status s = candidate_fits(m, candidate, &fits);
  if (s != WAVERNN_OK) return s;
  if (!fits) return fail(WAVERNN_E_INVALID, "placement %d does not fit the device", candidate);
  PersistPlan P;
  candidate_plan(m, candidate, &P);
  m->solo_hx = P.hx;
  m->solo_uxm = P.uxm;
  return WAVERNN_OK;
}

wavernn_status wavernn_tune(wavernn_model* m, int64_t n_steps, int32_t rounds, float* us_out, int32_t* chosen,
                            void* stream) {
  if (!m || n_steps < 16 || n_steps > ((int64_t)1 << 20) || rounds < 1 || rounds > 16)
    return fail(WAVERNN_E_INVALID, "bad tune arguments");
  if (chosen) *chosen = -1;
  if (us_out)
    for (int i = 0; i < 64; ++i) us_out[i] = -1.0f;
  if (m->path != PATH_PERSIST) return WAVERNN_OK;
  hipStream_t st = (hipStream_t)stream;
  bool fits[64];
  for (int i = 0; i < 64; ++i) {
    wavernn_status s = candidate_fits(m, i, &fits[i]);
    if (s != WAVERNN_OK) return s;
  }
  // one utterance of zero conditioning frames; a fused launch makes 2 samples a step
  const int64_t T = m->fused ? 2 * n_steps : n_steps;
  const int Dc = m->cfg.cond_dim, frame_len = m->cfg.frame_len > 0 ? m->cfg.frame_len : 1;
  const int64_t n_frames = Dc > 0 ? (T - 1) / frame_len + 1 : 0;
  const int64_t steps = m->fused ? n_steps + m->cfg.future_horizon + 1 : n_steps;
  float* cond = nullptr;
  uint16_t* out = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  const int hx0 = m->solo_hx, uxm0 = m->solo_uxm;
  u64* trace = m->trace;
  float best[64];
  for (int i = 0; i < 64; ++i) best[i] = 1e30f;
  wavernn_status s = WAVERNN_OK;
  auto step = [&](hipError_t e) {
    if (e != hipSuccess && s == WAVERNN_OK) s = fail(WAVERNN_E_HIP, "HIP error %s in wavernn_tune", hipGetErrorString(e));
    return s == WAVERNN_OK;
  };
  m->trace = nullptr;
  if (step(hipMalloc((void**)&out, (size_t)T * 2)) && (Dc == 0 || step(hipMalloc((void**)&cond, (size_t)n_frames * Dc * 4))) &&
      (Dc == 0 || step(hipMemsetAsync(cond, 0, (size_t)n_frames * Dc * 4, st))) &&
      step(hipEventCreate(&e0)) && step(hipEventCreate(&e1))) {
    RunIO io{1, T, cond, n_frames, 1, nullptr, nullptr, nullptr, out, nullptr, nullptr, nullptr, st};
    // round -1 warms up (code objects, tables) on the default placement
    for (int r = -1; r < rounds && s == WAVERNN_OK; ++r)
      for (int i = 0; i < 64 && s == WAVERNN_OK; ++i) {
        if (!fits[i] || (r < 0 && i > 0)) continue;
        PersistPlan P;
        candidate_plan(m, i, &P);
        m->solo_hx = P.hx;
        m->solo_uxm = P.uxm;
        if (!step(hipEventRecord(e0, st))) break;
        if ((s = run_persist(m, io)) != WAVERNN_OK) break;
        float ms = 0.0f;
        if (!step(hipEventRecord(e1, st)) || !step(hipEventSynchronize(e1)) || !step(hipEventElapsedTime(&ms, e0, e1))) break;
        unsigned err = 0;
        if (!step(hipMemcpy(&err, m->d_err, 4, hipMemcpyDeviceToHost))) break;
        if (err) {   // a wait expired: the candidate is out (the default placement is not)
          if (!step(hipMemset(m->d_err, 0, 64))) break;
          if (i == 0) s = fail(WAVERNN_E_DEVICE, "a bounded wait expired in a launch of the default placement");
          fits[i] = false;
          continue;
        }
        if (r >= 0) best[i] = std::min(best[i], ms * 1000.0f / (float)steps);
      }
  }
  m->trace = trace;
  m->solo_hx = hx0;
  m->solo_uxm = uxm0;
  if (s == WAVERNN_OK) {
    int k = 0;
    for (int i = 0; i < 64; ++i)
      if (fits[i] && best[i] < best[k]) k = i;
    if (us_out)
      for (int i = 0; i < 64; ++i) us_out[i] = fits[i] ? best[i] : -1.0f;
    PersistPlan P;
    candidate_plan(m, k, &P);
    m->solo_hx = P.hx;
    m->solo_uxm = P.uxm;
    if (chosen) *chosen = k;
  }
  // clean-up: the first failure is the one reported
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  const hipError_t se = hipStreamSynchronize(st);
  if (s == WAVERNN_OK && se != hipSuccess)
    s = fail(WAVERNN_E_HIP, "hipStreamSynchronize: %s", hipGetErrorString(se));
  if (out) (void)hipFree(out);
  if (cond) (void)hipFree(cond);
  return s;
}

wavernn_status wavernn_set_trace(wavernn_model* m, uint64_t* trace_dev, int64_t max_steps) {
  if (!m || max_steps < 0 || (max_steps > 0 && !trace_dev)) return fail(WAVERNN_E_INVALID, "bad trace arguments");
  m->trace = max_steps > 0 ? (u64*)trace_dev : nullptr;
  m->trace_steps = max_steps;
  return WAVERNN_OK;
}

wavernn_status wavernn_ctx_cnn_run(wavernn_model* m, int32_t n_streams, int64_t n_samples, const uint16_t* seq_dev,
                                   float* out_dev, void* stream) {
  if (!m) return fail(WAVERNN_E_INVALID, "null model");
  if (!m->has_cnn) return fail(WAVERNN_E_INVALID, "the model has no conditioning CNN");
  const int B = m->cfg.subscale;
  if (n_streams < 1 || n_streams > m->cfg.max_streams || n_samples < 0 || n_samples % B || n_samples / B > (1 << 26))
    return fail(WAVERNN_E_INVALID, "n_streams %d / n_samples %lld: bad sizes", n_streams, (long long)n_samples);
  if (n_samples == 0) return WAVERNN_OK;
  if (!seq_dev || !out_dev) return fail(WAVERNN_E_INVALID, "null buffer");
  const int64_t rows = n_samples / B;
  return run_cnn(m, n_streams, seq_dev, n_samples, (int)rows, 0, 0, rows, 0, out_dev, (hipStream_t)stream);
}

const char* wavernn_last_error(void) { return g_err.c_str(); }

}  // extern "C"
