// libjf C ABI: validation, buffer layout, weight packing and the launch
// sequence of one Jacobi iteration (see include/jf.h for the contract).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/jf.h"
#include "jf_internal.h"

using namespace jf;

// ---- errors ------------------------------------------------------------------------
static thread_local std::string g_err;

static jf_status fail(jf_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess)                                                               \
      return fail(JF_E_HIP, "%s: %s (%s:%d)", #expr, hipGetErrorString(e_), __FILE__, __LINE__); \
  } while (0)

extern "C" const char* jf_last_error(void) { return g_err.c_str(); }

// ---- layout ------------------------------------------------------------------------
namespace {


size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

struct Layout {
  // element counts / byte offsets
  size_t esz;                      // element size of cfg.dtype
  int Rp;                          // max_rows rounded up to 16
  int qkv_rows;                    // (H + 2G) * hd
  int n_pages;                     // pages per layer
  // packed (bytes)
  size_t l_qkv, l_o, l_gu, l_down, l_an, l_fn, layer_bytes;
  size_t p_lm, p_final, p_embed, packed_bytes;
  // kv (bytes)
  size_t page_bytes, kv_layer_bytes, kv_bytes;
  // workspace (bytes)
  size_t w_state, w_h, w_xn, w_q, w_attn, w_act, w_opart, w_ml, w_lm, w_g, w_parent, w_pos,
      w_vis, w_cos, w_sin, w_pt, w_rowmap, w_result, w_kpart, w_kcount, w_ss, w_sync, ws_bytes;
};

jf_status check_config(const jf_config* c) {
  if (!c) return fail(JF_E_INVAL, "config is null");
  if (c->dtype != JF_F32 && c->dtype != JF_BF16) return fail(JF_E_DTYPE, "dtype %d unsupported", c->dtype);
  if (c->n_layers < 1 || c->d_model < 128 || c->n_heads < 1 || c->n_kv_heads < 1 || c->d_ffn < 128 ||
      c->vocab < 16)
    return fail(JF_E_SHAPE, "non-positive or too small dimension");
  if (c->d_model % 128 || c->d_ffn % 128) return fail(JF_E_SHAPE, "d_model and d_ffn must be multiples of 128");
  if (c->d_model > 4096) return fail(JF_E_SHAPE, "d_model must be at most 4096");
  if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128)
    return fail(JF_E_SHAPE, "head_dim must be 32, 64 or 128");
  if (c->n_heads % c->n_kv_heads) return fail(JF_E_SHAPE, "n_heads must be a multiple of n_kv_heads");
  if ((c->n_heads * c->head_dim) % 128) return fail(JF_E_SHAPE, "n_heads * head_dim must be a multiple of 128");
  if (c->vocab % 16) return fail(JF_E_SHAPE, "vocab must be a multiple of 16");
  if (c->max_rows < 1 || c->max_rows > kMaxRows) return fail(JF_E_SHAPE, "max_rows must be in [1, %d]", kMaxRows);
  if (c->max_ctx < 64 || c->max_ctx % 64) return fail(JF_E_SHAPE, "max_ctx must be a positive multiple of 64");
  if (!(c->rms_eps > 0.f) || !(c->rope_base > 1.f)) return fail(JF_E_INVAL, "rms_eps / rope_base out of range");
  return JF_OK;
}

Layout make_layout(const jf_config& c) {
  Layout L{};
  L.esz = c.dtype == JF_BF16 ? 2 : 4;
  L.Rp = (c.max_rows + 15) / 16 * 16;
  const size_t d = c.d_model, F = c.d_ffn, V = c.vocab, Hhd = (size_t)c.n_heads * c.head_dim;
  L.qkv_rows = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
  L.n_pages = c.max_ctx / kPage;
  size_t off = 0;
  L.l_qkv = off; off = align_up(off + (size_t)L.qkv_rows * d * L.esz);
  L.l_o = off; off = align_up(off + d * Hhd * L.esz);
  L.l_gu = off; off = align_up(off + 2 * F * d * L.esz);
  L.l_down = off; off = align_up(off + d * F * L.esz);
  L.l_an = off; off = align_up(off + d * 4);
  L.l_fn = off; off = align_up(off + d * 4);
  L.layer_bytes = off;
  off = L.layer_bytes * c.n_layers;
  L.p_lm = off; off = align_up(off + V * d * L.esz);
  L.p_final = off; off = align_up(off + d * 4);
  L.p_embed = off; off = align_up(off + V * d * L.esz);
  L.packed_bytes = off;

  L.page_bytes = (size_t)2 * c.n_kv_heads * kPage * c.head_dim * L.esz;
  L.kv_layer_bytes = L.page_bytes * L.n_pages;
  L.kv_bytes = L.kv_layer_bytes * c.n_layers;

  const size_t Rp = L.Rp;
  off = 0;
  L.w_state = off; off = align_up(off + 64);
  L.w_h = off; off = align_up(off + Rp * d * 4);
  // activations: two bf16 planes (hi, lo) for bf16 models, one fp32 plane
  // otherwise -- 4 bytes per element either way
  L.w_xn = off; off = align_up(off + Rp * d * 4);
  L.w_q = off; off = align_up(off + Rp * Hhd * 4);
  L.w_attn = off; off = align_up(off + Rp * Hhd * 4);
  L.w_act = off; off = align_up(off + Rp * F * 4);
  L.w_opart = off; off = align_up(off + (size_t)kAttnMaxSplits * Rp * c.n_heads * c.head_dim * 4);
  L.w_ml = off; off = align_up(off + (size_t)kAttnMaxSplits * Rp * c.n_heads * 2 * 4);
  L.w_lm = off; off = align_up(off + (V / 16) * Rp * 8);
  L.w_g = off; off = align_up(off + Rp * 4);
  L.w_parent = off; off = align_up(off + Rp * 4);
  L.w_pos = off; off = align_up(off + Rp * 4);
  L.w_vis = off; off = align_up(off + Rp * kVisWords * 8);
  L.w_cos = off; off = align_up(off + (size_t)c.max_ctx * (c.head_dim / 2) * 4);
  L.w_sin = off; off = align_up(off + (size_t)c.max_ctx * (c.head_dim / 2) * 4);
  L.w_pt = off; off = align_up(off + (size_t)L.n_pages * 4);
  size_t maxrows = std::max<size_t>({(size_t)L.qkv_rows, 2 * F, d, V});
  L.w_rowmap = off; off = align_up(off + maxrows * 4);
  L.w_result = off; off = align_up(off + 64);
  L.w_kpart = off; off = align_up(off + kGemmPartFloats * 4);
  L.w_kcount = off; off = align_up(off + kGemmCounters * 4);
  // RMSNorm sums of squares: two fixed-point accumulators of 3 word planes
  L.w_ss = off; off = align_up(off + 2 * 3 * Rp * 8);
  // flags and counters of the fused attention launch
  L.w_sync = off; off = align_up(off + kAttnBlockSyncWords * 4);
  L.ws_bytes = off;
  return L;
}

}  // namespace

struct jf_model {
  jf_config cfg;
  Layout L;
  char* packed;
  char* kv;
  char* ws;
  int C_ub;          // host upper bound of the committed length
  int last_rows;     // rows of the last step (0: no step to commit)
  int last_tree;     // last step was a multi-block step
  int fused_attention = 0;            // JF_OPT_FUSED_ATTENTION (measured slower; off by default)
  int n_cus = 0;                      // compute units of the model's device
  int attn_block_occ = 0;             // fused attention workgroups per compute unit
  uint32_t epoch = 0;                 // launches of the fused attention (never 0 once used)
  int prof_class = 0;                 // kernel class being timed (0: none)
  std::vector<hipEvent_t> prof_events;  // pairs (start, end), reused
  size_t prof_used = 0;
  int32_t* state() { return reinterpret_cast<int32_t*>(ws + L.w_state); }
  int32_t* flags() { return state() + 1; }
  template <typename P> P* at(size_t off) { return reinterpret_cast<P*>(ws + off); }
  char* layer(int l) { return packed + (size_t)l * L.layer_bytes; }
  char* kv_layer(int l) { return kv + (size_t)l * L.kv_layer_bytes; }
  Epi epi() {
    Epi e{};
    e.kpart = at<float>(L.w_kpart);
    e.kcount = at<int32_t>(L.w_kcount);
    return e;
  }
};

extern "C" jf_status jf_query_sizes(const jf_config* cfg, size_t* packed_bytes, size_t* kv_bytes,
                                    size_t* ws_bytes) {
  jf_status s = check_config(cfg);
  if (s != JF_OK) return s;
  if (!packed_bytes || !kv_bytes || !ws_bytes) return fail(JF_E_INVAL, "null output pointer");
  Layout L = make_layout(*cfg);
  *packed_bytes = L.packed_bytes;
  *kv_bytes = L.kv_bytes;
  *ws_bytes = L.ws_bytes;
  return JF_OK;
}

// Row order of the fused QKV matrix: q heads, k heads, v heads; inside every
// 16-row tile of a q/k head, rows 0..7 are dims 8t..8t+7 and rows 8..15 are
// dims hd/2+8t..hd/2+8t+7 so each RoPE pair (i, i + hd/2) sits in one tile.
static std::vector<int32_t> qkv_rowmap(const jf_config& c) {
  std::vector<int32_t> m;
  const int hd = c.head_dim, half = hd / 2;
  auto add_head = [&](int src, int head, bool rope) {
    for (int w = 0; w < hd; ++w) {
      int dim = w;
      if (rope) {
        int t = w / 16, cc = w % 16;
        dim = cc < 8 ? 8 * t + cc : half + 8 * t + (cc - 8);
      }
      m.push_back((src << 24) | (head * hd + dim));
    }
  };
  for (int h = 0; h < c.n_heads; ++h) add_head(0, h, true);
  for (int h = 0; h < c.n_kv_heads; ++h) add_head(1, h, true);
  for (int h = 0; h < c.n_kv_heads; ++h) add_head(2, h, false);
  return m;
}

// gate/up interleaved by 16-row tiles: tile 2t = gate rows 16t.., 2t+1 = up rows 16t..
static std::vector<int32_t> gateup_rowmap(const jf_config& c) {
  std::vector<int32_t> m;
  for (int t = 0; t < c.d_ffn / 16; ++t) {
    for (int i = 0; i < 16; ++i) m.push_back((0 << 24) | (16 * t + i));
    for (int i = 0; i < 16; ++i) m.push_back((1 << 24) | (16 * t + i));
  }
  return m;
}

extern "C" jf_status jf_model_load(const jf_config* cfg, const void* const* d_weights,
                                   int32_t n_weights, void* d_packed, void* d_kv, void* d_ws,
                                   jf_stream stream, jf_model** out) {
  jf_status s = check_config(cfg);
  if (s != JF_OK) return s;
  if (!d_weights || !d_packed || !d_kv || !d_ws || !out) return fail(JF_E_INVAL, "null pointer argument");
  if (n_weights != 3 + 9 * cfg->n_layers)
    return fail(JF_E_INVAL, "n_weights = %d, expected %d", n_weights, 3 + 9 * cfg->n_layers);
  for (int i = 0; i < n_weights; ++i)
    if (!d_weights[i]) return fail(JF_E_INVAL, "weight %d is null", i);
  *out = nullptr;
  hipStream_t st = (hipStream_t)stream;
  jf_model* m = new (std::nothrow) jf_model();
  if (!m) return fail(JF_E_INVAL, "out of host memory");
  m->cfg = *cfg;
  m->L = make_layout(*cfg);
  m->packed = (char*)d_packed;
  m->kv = (char*)d_kv;
  m->ws = (char*)d_ws;
  const jf_config& c = *cfg;
  const Layout& L = m->L;
  const int dt = c.dtype;
  const int d = c.d_model, F = c.d_ffn, V = c.vocab, Hhd = c.n_heads * c.head_dim;

  auto bail = [&](jf_status st_) { delete m; return st_; };
#define LOAD_TRY(expr)                                                                      \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return bail(fail(JF_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)));                 \
  } while (0)

  // Host tables: rope cos/sin (float64 math, rounded to float32), page table.
  const int half = c.head_dim / 2;
  std::vector<float> cs((size_t)c.max_ctx * half), sn((size_t)c.max_ctx * half);
  for (int p = 0; p < c.max_ctx; ++p)
    for (int i = 0; i < half; ++i) {
      double inv = std::pow((double)c.rope_base, -(2.0 * i) / c.head_dim);
      double ang = (double)p * inv;
      cs[(size_t)p * half + i] = (float)std::cos(ang);
      sn[(size_t)p * half + i] = (float)std::sin(ang);
    }
  std::vector<int32_t> pt(L.n_pages);
  for (int i = 0; i < L.n_pages; ++i) pt[i] = i;
  std::vector<int32_t> rm_qkv = qkv_rowmap(c), rm_gu = gateup_rowmap(c);

  LOAD_TRY(hipMemsetAsync(d_kv, 0, L.kv_bytes, st));
  LOAD_TRY(hipMemsetAsync(m->ws + L.w_state, 0, 64, st));
  LOAD_TRY(hipMemsetAsync(m->ws + L.w_kcount, 0, kGemmCounters * 4, st));
  LOAD_TRY(hipMemsetAsync(m->ws + L.w_sync, 0, kAttnBlockSyncWords * 4, st));
  {
    int dev = 0;
    LOAD_TRY(hipGetDevice(&dev));
    LOAD_TRY(hipDeviceGetAttribute(&m->n_cus, hipDeviceAttributeMultiprocessorCount, dev));
    m->attn_block_occ = attn_block_occupancy(c.head_dim);
  }
  LOAD_TRY(hipMemcpyAsync(m->ws + L.w_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, st));
  LOAD_TRY(hipMemcpyAsync(m->ws + L.w_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice, st));
  LOAD_TRY(hipMemcpyAsync(m->ws + L.w_pt, pt.data(), pt.size() * 4, hipMemcpyHostToDevice, st));

  int32_t* rowmap = m->at<int32_t>(L.w_rowmap);
  const size_t esz = L.esz;
  // embedding (natural layout) and the LM head / final norm
  LOAD_TRY(hipMemcpyAsync(m->packed + L.p_embed, d_weights[0], (size_t)V * d * esz,
                          hipMemcpyDeviceToDevice, st));
  const int base_final = 1 + 9 * c.n_layers;
  LOAD_TRY(launch_to_f32(dt, d_weights[base_final], (float*)(m->packed + L.p_final), d, st));
  {
    const void* src[1] = {d_weights[base_final + 1]};
    LOAD_TRY(launch_pack(dt, V, d, src, 1, nullptr, m->packed + L.p_lm, st));
  }
  for (int l = 0; l < c.n_layers; ++l) {
    const void* const* w = d_weights + 1 + 9 * l;
    char* lp = m->layer(l);
    LOAD_TRY(launch_to_f32(dt, w[0], (float*)(lp + L.l_an), d, st));
    LOAD_TRY(launch_to_f32(dt, w[5], (float*)(lp + L.l_fn), d, st));
    LOAD_TRY(hipMemcpyAsync(rowmap, rm_qkv.data(), rm_qkv.size() * 4, hipMemcpyHostToDevice, st));
    const void* qkv[3] = {w[1], w[2], w[3]};
    LOAD_TRY(launch_pack(dt, L.qkv_rows, d, qkv, 3, rowmap, lp + L.l_qkv, st));
    const void* o[1] = {w[4]};
    LOAD_TRY(launch_pack(dt, d, Hhd, o, 1, nullptr, lp + L.l_o, st));
    LOAD_TRY(hipStreamSynchronize(st));  // rowmap reused below
    LOAD_TRY(hipMemcpyAsync(rowmap, rm_gu.data(), rm_gu.size() * 4, hipMemcpyHostToDevice, st));
    const void* gu[2] = {w[6], w[7]};
    LOAD_TRY(launch_pack(dt, 2 * F, d, gu, 2, rowmap, lp + L.l_gu, st));
    const void* dn[1] = {w[8]};
    LOAD_TRY(launch_pack(dt, d, F, dn, 1, nullptr, lp + L.l_down, st));
    LOAD_TRY(hipStreamSynchronize(st));
  }
  LOAD_TRY(hipStreamSynchronize(st));
#undef LOAD_TRY
  m->C_ub = 0;
  m->last_rows = 0;
  m->last_tree = 0;
  *out = m;
  return JF_OK;
}

extern "C" jf_status jf_model_free(jf_model* m) {
  if (!m) return fail(JF_E_INVAL, "model is null");
  for (hipEvent_t e : m->prof_events) (void)hipEventDestroy(e);
  delete m;
  return JF_OK;
}

// Records an event on st if kernel class cls is being timed.
static jf_status prof_mark(jf_model* m, int cls, hipStream_t st) {
  if (m->prof_class != cls) return JF_OK;
  if (m->prof_used == m->prof_events.size()) {
    // Timing only (read after a stream synchronisation): no system-scope
    // fence, whose cache writeback would be counted in the kernel's time.
    hipEvent_t e;
    HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
    m->prof_events.push_back(e);
  }
  HIP_TRY(hipEventRecord(m->prof_events[m->prof_used++], st));
  return JF_OK;
}
#define PROF(cls)                                   \
  do {                                              \
    jf_status ps_ = prof_mark(m, (cls), st);        \
    if (ps_ != JF_OK) return ps_;                   \
  } while (0)

extern "C" jf_status jf_model_set_option(jf_model* m, int32_t option, int32_t value) {
  if (!m) return fail(JF_E_INVAL, "model is null");
  if (option != JF_OPT_FUSED_ATTENTION) return fail(JF_E_INVAL, "unknown option %d", option);
  if (value != 0 && value != 1) return fail(JF_E_INVAL, "option %d takes 0 or 1, got %d", option, value);
  m->fused_attention = value;
  return JF_OK;
}

extern "C" jf_status jf_profile_begin(jf_model* m, int32_t kernel_class) {
  if (!m) return fail(JF_E_INVAL, "model is null");
  if (kernel_class < JF_KERNEL_QKV || kernel_class > JF_KERNEL_ATTN_BLOCK)
    return fail(JF_E_INVAL, "unknown kernel class %d", kernel_class);
  m->prof_class = kernel_class;
  m->prof_used = 0;
  return JF_OK;
}

extern "C" jf_status jf_profile_end(jf_model* m, double* total_ms, int32_t* launches) {
  if (!m || !total_ms || !launches) return fail(JF_E_INVAL, "null pointer argument");
  if (m->prof_class == 0) return fail(JF_E_STATE, "no profile in progress");
  double t = 0.0;
  for (size_t i = 0; i + 1 < m->prof_used; i += 2) {
    HIP_TRY(hipEventSynchronize(m->prof_events[i + 1]));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, m->prof_events[i], m->prof_events[i + 1]));
    t += ms;
  }
  *total_ms = t;
  *launches = (int32_t)(m->prof_used / 2);
  m->prof_class = 0;
  m->prof_used = 0;
  return JF_OK;
}

// ---- projections ----------------------------------------------------------------------
// Compute units of the current device (looked up once).
static int device_cus() {
  static int cus = 0;
  if (!cus) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) ==
                                                 hipSuccess)
      cus = n;
  }
  return cus > 0 ? cus : 256;
}

// One projection Y[R][N] = X[R][K] W^T with epilogue ep: the column-slice
// kernel (gemm_mr.hip) for bf16 where its plan takes the shape (more than
// 32 rows: wide matrices and long-K narrow ones), else the weight-streaming
// kernel.  *part_blocks (if not null) gets the number of per-row argmax key
// slots the launch writes (EPI_ARGMAX).  split_k = false keeps K in one
// workgroup (callers without split-K scratch).
static hipError_t run_gemm(int dtype, int R, int N, int K, const void* X, size_t xplane, const void* W, const Epi& ep,
                           hipStream_t st, int* part_blocks = nullptr, bool split_k = true) {
  if (dtype == JF_BF16 && ep.row0 == 0) {
    MrPlan mp{};
    if (gemm_mr_plan(mp, R, N, K, ep.kind, device_cus(), split_k ? 64 : 1)) {
      if (part_blocks) *part_blocks = gemm_mr_part_blocks(mp);
      return launch_gemm_mr(X, xplane, W, mp, ep, st);
    }
  }
  GemmShape gs{R, N, K, 1, 1, 1};
  gemm_plan(gs, ep.kind);
  if (!split_k) gs.S = 1;
  else gemm_tail_split(gs, device_cus());
  if (part_blocks) *part_blocks = (int)gemm_blocks(gs);
  return launch_gemm(dtype, X, xplane, W, gs, ep, st);
}

// ---- forward pass of one step ---------------------------------------------------------
// Runs rows through all layers; the K/V of row r land in cache slot C + r.
// lm: 0 = no LM head, 1 = all rows, 2 = last row only.  g receives the argmax.
// The rows' forest comes from sg, or from the packed layout when pk is set.
struct PackedSpec {
  int n_blocks, n, mask;
};
// lm_parts (lm == 1): when not null, the argmax reduction is left to the
// caller's fused tail, which gets the number of per-block key slots here.
static jf_status forward(jf_model* m, const int32_t* d_tokens, int R, const SegArgs& sg, int lm,
                         int32_t* d_g, float* d_logits, hipStream_t st, const PackedSpec* pk = nullptr,
                         int* lm_parts = nullptr) {
  const jf_config& c = m->cfg;
  const Layout& L = m->L;
  const int dt = c.dtype;
  const int d = c.d_model, F = c.d_ffn, H = c.n_heads, G = c.n_kv_heads, hd = c.head_dim;
  const int Hhd = H * hd;
  int32_t* state = m->state();
  float* h = m->at<float>(L.w_h);
  void* xn = m->ws + L.w_xn;
  int32_t* pos = m->at<int32_t>(L.w_pos);

  if (pk)
    HIP_TRY(launch_tree_packed(pk->n_blocks, pk->n, pk->mask, state, m->flags(), m->at<int32_t>(L.w_parent),
                               pos, m->at<uint64_t>(L.w_vis), st));
  else
    HIP_TRY(launch_tree(sg, R, state, m->flags(), m->at<int32_t>(L.w_parent), pos,
                        m->at<uint64_t>(L.w_vis), st));
  const size_t Rp = L.Rp;
  const size_t pl_d = Rp * d, pl_h = Rp * Hhd, pl_f = Rp * F;  // activation plane strides
  // The RMSNorms are folded into the projections.  Every residual add writes
  // xn = h * (next gain) and adds the rows' sums of squares into one of two
  // accumulators; the next projection scales its output rows by 1 / rms.
  // ss_a feeds the QKV projections and the LM head, ss_f the gate/up ones;
  // each producer zeroes the accumulator it does not fill (already consumed).
  uint64_t* ss_a = m->at<uint64_t>(L.w_ss);
  uint64_t* ss_f = ss_a + 3 * Rp;
  const int ss_stride = (int)Rp;
  auto norm_in = [&](Epi& ep, const uint64_t* ss) {
    ep.ss_in = ss; ep.ss_stride = ss_stride; ep.norm_inv_d = 1.0 / d; ep.norm_eps = c.rms_eps;
  };
  auto norm_out = [&](Epi& ep, const float* gain, uint64_t* ss, uint64_t* clear) {
    ep.gain_next = gain; ep.xg = xn; ep.xg_plane = pl_d; ep.ss_out = ss; ep.ss_clear = clear;
    ep.ss_stride = ss_stride;
  };
  HIP_TRY(launch_embed(dt, d_tokens, R, m->packed + L.p_embed, (const float*)(m->layer(0) + L.l_an), d,
                       c.vocab, h, xn, pl_d, ss_a, ss_f, ss_stride, m->flags(), st));
  const int keys_ub = std::min(m->C_ub + R, c.max_ctx);
  // The attention half of every layer as one persistent launch (layer.hip)
  // when the step qualifies; its plan is the same for all layers.
  SideArgs sa{};
  bool fused = m->fused_attention && dt == JF_BF16 && hd == 128 && R <= kAttnBlockMaxRows &&
               m->attn_block_occ >= 1 && m->n_cus >= 1 && Hhd <= 4096 && d <= 4096 &&
               m->L.qkv_rows / 16 <= kAttnBlockMaxTiles;
  if (fused) {
    sa.R = R; sa.d = d; sa.H = H; sa.G = G; sa.hd = hd; sa.max_ctx = c.max_ctx;
    sa.qkv_tiles = m->L.qkv_rows / 16; sa.o_tiles = d / 16;
    sa.kc_qkv = d / 128; sa.kc_o = Hhd / 128;
    sa.p_qkv = pack_group(m->L.qkv_rows); sa.p_o = pack_group(d);
    sa.keys_ub = keys_ub;
    attn_block_plan(sa);
    fused = sa.G * sa.qtiles <= kAttnBlockMaxGT && sa.splits <= kAttnMaxSplits && sa.kc_o <= 32;
  }
  for (int l = 0; l < c.n_layers; ++l) {
    char* lp = m->layer(l);
    if (fused) {
      sa.x = xn; sa.x_plane = pl_d; sa.w_qkv = lp + L.l_qkv;
      sa.ss_in = ss_a; sa.ss_stride = ss_stride; sa.norm_inv_d = 1.0 / d; sa.norm_eps = c.rms_eps;
      sa.q = m->ws + L.w_q; sa.q_plane = pl_h; sa.kv = m->kv_layer(l);
      sa.page_table = m->at<int32_t>(L.w_pt); sa.pos = pos; sa.state = state;
      sa.rope_cos = m->at<float>(L.w_cos); sa.rope_sin = m->at<float>(L.w_sin); sa.flags = m->flags();
      sa.vis = m->at<uint64_t>(L.w_vis);
      sa.o_part = m->at<float>(L.w_opart); sa.ml_part = m->at<float>(L.w_ml);
      sa.attn = m->ws + L.w_attn; sa.attn_plane = pl_h;
      sa.w_o = lp + L.l_o; sa.h = h; sa.gain_next = (const float*)(lp + L.l_fn);
      sa.xg = xn; sa.xg_plane = pl_d; sa.ss_out = ss_f; sa.ss_clear = ss_a;
      sa.sync = m->at<uint32_t>(L.w_sync);
      if (++m->epoch == 0) ++m->epoch;
      sa.epoch = m->epoch;
      PROF(JF_KERNEL_ATTN_BLOCK);
      HIP_TRY(launch_attn_block(sa, m->n_cus, st));
      PROF(JF_KERNEL_ATTN_BLOCK);
    }
    // a3: attention RMSNorm (folded) + QKV + RoPE + K/V into the cache slots C + r
    if (!fused) {
      Epi ep = m->epi();
      ep.kind = EPI_QKV; ep.R = R;
      norm_in(ep, ss_a);
      ep.q = m->ws + L.w_q; ep.q_plane = pl_h; ep.kv = m->kv_layer(l);
      ep.page_table = m->at<int32_t>(L.w_pt);
      ep.pos = pos; ep.state = state; ep.rope_cos = m->at<float>(L.w_cos); ep.rope_sin = m->at<float>(L.w_sin);
      ep.H = H; ep.G = G; ep.hd = hd; ep.max_ctx = c.max_ctx; ep.flags = m->flags();
      PROF(JF_KERNEL_QKV);
      HIP_TRY(run_gemm(dt, R, m->L.qkv_rows, d, xn, pl_d, lp + L.l_qkv, ep, st));
      PROF(JF_KERNEL_QKV);
    }
    // a4: attention
    if (!fused) {
      AttnArgs a{};
      a.H = H; a.G = G; a.hd = hd; a.R = R; a.max_ctx = c.max_ctx; a.keys_ub = keys_ub;
      a.lds_ok = dt == JF_BF16;
      attn_plan(a);
      a.q = m->ws + L.w_q; a.q_plane = pl_h; a.kv = m->kv_layer(l); a.page_table = m->at<int32_t>(L.w_pt);
      a.state = state; a.vis = m->at<uint64_t>(L.w_vis);
      a.o_part = m->at<float>(L.w_opart); a.ml_part = m->at<float>(L.w_ml); a.out = m->ws + L.w_attn;
      a.out_plane = pl_h;
      PROF(JF_KERNEL_ATTN);
      HIP_TRY(launch_attention(dt, a, st));
      PROF(JF_KERNEL_ATTN);
    }
    // a5: O projection + residual, writing the FFN RMSNorm's input
    if (!fused) {
      Epi ep = m->epi();
      ep.kind = EPI_RESID; ep.R = R; ep.f32 = h; ep.ldf = d;
      norm_out(ep, (const float*)(lp + L.l_fn), ss_f, ss_a);
      PROF(JF_KERNEL_O);
      HIP_TRY(run_gemm(dt, R, d, Hhd, m->ws + L.w_attn, pl_h, lp + L.l_o, ep, st));
      PROF(JF_KERNEL_O);
    }
    // a6: FFN RMSNorm (folded), gate/up + SwiGLU, down + residual
    {
      Epi ep = m->epi();
      ep.kind = EPI_SWIGLU; ep.R = R; ep.act = m->ws + L.w_act; ep.act_k = F; ep.act_plane = pl_f;
      norm_in(ep, ss_f);
      PROF(JF_KERNEL_GATEUP);
      HIP_TRY(run_gemm(dt, R, 2 * F, d, xn, pl_d, lp + L.l_gu, ep, st));
      PROF(JF_KERNEL_GATEUP);
    }
    // down projection + residual, writing the next RMSNorm's input (the next
    // layer's attention norm, or the final norm before the LM head)
    {
      Epi ep = m->epi();
      ep.kind = EPI_RESID; ep.R = R; ep.f32 = h; ep.ldf = d;
      if (l + 1 < c.n_layers)
        norm_out(ep, (const float*)(m->layer(l + 1) + L.l_an), ss_a, ss_f);
      else if (lm != 0)
        norm_out(ep, (const float*)(m->packed + L.p_final), ss_a, ss_f);
      PROF(JF_KERNEL_DOWN);
      HIP_TRY(run_gemm(dt, R, d, F, m->ws + L.w_act, pl_f, lp + L.l_down, ep, st));
      PROF(JF_KERNEL_DOWN);
    }
  }
  if (lm == 0) return JF_OK;
  // a7: final RMSNorm (folded) + LM head with fused argmax (logits optional);
  // lm == 2 reads only the last row
  const int Rl = lm == 2 ? 1 : R;
  Epi ep = m->epi();
  ep.kind = EPI_ARGMAX; ep.R = Rl; ep.part = m->at<uint64_t>(L.w_lm); ep.part_stride = L.Rp;
  ep.logits = d_logits; ep.ldl = c.vocab;
  ep.row0 = lm == 2 ? R - 1 : 0;
  norm_in(ep, ss_a);
  PROF(JF_KERNEL_LMHEAD);
  int part_blocks = 0;
  HIP_TRY(run_gemm(dt, Rl, c.vocab, d, xn, pl_d, m->packed + L.p_lm, ep, st, &part_blocks));
  PROF(JF_KERNEL_LMHEAD);
  if (lm_parts) {
    *lm_parts = part_blocks;
    return JF_OK;
  }
  HIP_TRY(launch_argmax_reduce(ep.part, part_blocks, L.Rp, Rl, d_g, st));
  return JF_OK;
}

// Capacity check against the host's upper bound of C.  The bound only grows
// by the rows of each committed step (the accepted count stays on the
// device); when it would exceed max_ctx the exact C is read back (one stream
// synchronisation) before refusing.
static jf_status check_rows(jf_model* m, int R, hipStream_t st) {
  if (R < 1 || R > m->cfg.max_rows)
    return fail(JF_E_CAPACITY, "rows %d outside [1, max_rows=%d]", R, m->cfg.max_rows);
  if (m->C_ub + R > m->cfg.max_ctx) {
    int32_t v = 0;
    HIP_TRY(hipMemcpyAsync(&v, m->state(), 4, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    m->C_ub = v;
  }
  if (m->C_ub + R > m->cfg.max_ctx)
    return fail(JF_E_CAPACITY, "committed length %d + rows %d exceeds max_ctx %d", m->C_ub, R,
                m->cfg.max_ctx);
  return JF_OK;
}

extern "C" jf_status jf_prefill(jf_model* m, const int32_t* d_tokens, int32_t n, int32_t* d_pending,
                                jf_stream stream) {
  if (!m || !d_tokens || !d_pending) return fail(JF_E_INVAL, "null pointer argument");
  if (m->C_ub != 0) return fail(JF_E_STATE, "prefill needs an empty cache (truncate to 0 first)");
  if (n < 1 || n > m->cfg.max_ctx) return fail(JF_E_CAPACITY, "prompt length %d outside [1, max_ctx]", n);
  hipStream_t st = (hipStream_t)stream;
  const int chunk = m->cfg.max_rows;
  for (int s = 0; s < n; s += chunk) {
    const int R = std::min(chunk, n - s);
    SegArgs sg{};
    sg.n = 1; sg.first[0] = 0; sg.nrows[0] = R; sg.attach[0] = -1; sg.role[0] = 0; sg.verify_from[0] = 1;
    const bool last = s + R == n;
    jf_status r = forward(m, d_tokens + s, R, sg, last ? 2 : 0, d_pending, nullptr, st);
    if (r != JF_OK) return r;
    HIP_TRY(launch_commit(m->cfg.dtype, m->kv, m->cfg.n_layers, m->L.n_pages, m->cfg.n_kv_heads,
                          m->cfg.head_dim, m->at<int32_t>(m->L.w_pt), m->state(), nullptr,
                          m->at<int32_t>(m->L.w_result), 0, R, m->cfg.max_ctx, st));
    m->C_ub += R;
  }
  m->last_rows = 0;
  return JF_OK;
}

extern "C" jf_status jf_jacobi_step(jf_model* m, const int32_t* d_draft, int32_t n, int32_t mode,
                                    uint64_t pad_seed, int32_t* d_argmax, jf_step_result* d_result,
                                    int32_t* d_next_draft, float* d_logits, jf_stream stream) {
  if (!m || !d_draft || !d_argmax || !d_result || !d_next_draft)
    return fail(JF_E_INVAL, "null pointer argument");
  if (mode < 0 || mode > (1 | JF_STEP_COMMIT))
    return fail(JF_E_INVAL, "mode must be 0 (block) or 1 (window), optionally | JF_STEP_COMMIT");
  if (m->C_ub == 0) return fail(JF_E_STATE, "empty cache: prefill the prompt first");
  hipStream_t st = (hipStream_t)stream;
  jf_status s = check_rows(m, n, st);
  if (s != JF_OK) return s;
  const int commit = (mode & JF_STEP_COMMIT) ? 1 : 0;
  SegArgs sg{};
  sg.n = 1; sg.first[0] = 0; sg.nrows[0] = n; sg.attach[0] = -1; sg.role[0] = 0; sg.verify_from[0] = 1;
  PROF(JF_KERNEL_STEP);
  int parts = 0;
  s = forward(m, d_draft, n, sg, 1, d_argmax, d_logits, st, nullptr, &parts);
  if (s != JF_OK) return s;
  HIP_TRY(launch_argmax_accept_linear(m->at<uint64_t>(m->L.w_lm), parts, m->L.Rp, d_draft, n, mode & 1, pad_seed,
                                      m->cfg.vocab, m->state(), m->flags(), reinterpret_cast<int32_t*>(d_result),
                                      d_next_draft, d_argmax, commit, m->cfg.max_ctx, st));
  PROF(JF_KERNEL_STEP);
  if (commit) {
    m->C_ub = std::min(m->C_ub + n, m->cfg.max_ctx);
    m->last_rows = 0;
  } else {
    m->last_rows = n;
  }
  m->last_tree = 0;
  return JF_OK;
}

static jf_status check_segments(const jf_segment* segs, int n_segs, int R, SegArgs* out) {
  if (!segs) return fail(JF_E_INVAL, "segments are null");
  if (n_segs < 1 || n_segs > JF_MAX_SEGMENTS)
    return fail(JF_E_INVAL, "n_segs %d outside [1, %d]", n_segs, JF_MAX_SEGMENTS);
  int next = 0;
  for (int i = 0; i < n_segs; ++i) {
    const jf_segment& s = segs[i];
    if (s.first_row != next || s.n_rows < 1)
      return fail(JF_E_INVAL, "segment %d does not continue the row order", i);
    if (s.attach_row < -1 || s.attach_row >= s.first_row)
      return fail(JF_E_INVAL, "segment %d must attach to an earlier row or -1", i);
    if (s.role < JF_ROLE_RA || s.role > JF_ROLE_PSEUDO)
      return fail(JF_E_INVAL, "segment %d has an unknown role", i);
    if (s.verify_from < 0 || s.verify_from > s.n_rows)
      return fail(JF_E_INVAL, "segment %d verify_from outside [0, n_rows]", i);
    if (i > 0 && s.role == JF_ROLE_RA) return fail(JF_E_INVAL, "only segment 0 may be real-active");
    next += s.n_rows;
    out->first[i] = s.first_row; out->nrows[i] = s.n_rows; out->attach[i] = s.attach_row;
    out->role[i] = s.role; out->verify_from[i] = s.verify_from;
  }
  if (next != R) return fail(JF_E_INVAL, "segments cover %d rows, R = %d", next, R);
  if (segs[0].attach_row != -1 || segs[0].role != JF_ROLE_RA || segs[0].verify_from != 1)
    return fail(JF_E_INVAL, "segment 0 must be the real-active draft (attach -1, verify_from 1)");
  out->n = n_segs;
  return JF_OK;
}

extern "C" jf_status jf_multiblock_step(jf_model* m, const int32_t* d_tokens, int32_t R,
                                        const jf_segment* segs, int32_t n_segs, int32_t* d_argmax,
                                        int32_t* d_seg_accept, jf_step_result* d_result,
                                        int32_t* d_path, float* d_logits, jf_stream stream) {
  if (!m || !d_tokens || !d_argmax || !d_seg_accept || !d_result || !d_path)
    return fail(JF_E_INVAL, "null pointer argument");
  if (m->C_ub == 0) return fail(JF_E_STATE, "empty cache: prefill the prompt first");
  hipStream_t st = (hipStream_t)stream;
  SegArgs sg{};
  jf_status s = check_segments(segs, n_segs, R, &sg);
  if (s != JF_OK) return s;
  s = check_rows(m, R, st);
  if (s != JF_OK) return s;
  PROF(JF_KERNEL_STEP);
  int parts = 0;
  s = forward(m, d_tokens, R, sg, 1, d_argmax, d_logits, st, nullptr, &parts);
  if (s != JF_OK) return s;
  HIP_TRY(launch_argmax_accept_tree(m->at<uint64_t>(m->L.w_lm), parts, m->L.Rp, sg, d_tokens, R,
                                    m->at<int32_t>(m->L.w_parent), m->state(), m->flags(), d_seg_accept,
                                    reinterpret_cast<int32_t*>(d_result), d_path, d_argmax, st));
  PROF(JF_KERNEL_STEP);
  m->last_rows = R;
  m->last_tree = 1;
  return JF_OK;
}

static_assert(kMaxRows == JF_MAX_ROWS && kVisWords == JF_VIS_WORDS, "row limits of jf.h");
static_assert(kMaskNoisyContext == JF_MASK_NOISY_CONTEXT && kMaskCleanContext == JF_MASK_CLEAN_CONTEXT,
              "mask constants");

extern "C" jf_status jf_packed_forward(jf_model* m, const int32_t* d_tokens, int32_t n_blocks, int32_t n,
                                       int32_t mask, int32_t* d_argmax, float* d_logits, jf_stream stream) {
  if (!m || !d_tokens || !d_argmax) return fail(JF_E_INVAL, "null pointer argument");
  if (mask != JF_MASK_NOISY_CONTEXT && mask != JF_MASK_CLEAN_CONTEXT)
    return fail(JF_E_INVAL, "mask must be JF_MASK_NOISY_CONTEXT or JF_MASK_CLEAN_CONTEXT");
  if (n_blocks < 1 || n < 1) return fail(JF_E_SHAPE, "need n_blocks >= 1 and n >= 1");
  if (m->C_ub == 0) return fail(JF_E_STATE, "empty cache: prefill the prompt first");
  if ((long long)2 * n_blocks * n > m->cfg.max_rows)
    return fail(JF_E_CAPACITY, "2 * n_blocks * n = %lld rows exceeds max_rows %d", (long long)2 * n_blocks * n,
                m->cfg.max_rows);
  const int R = 2 * n_blocks * n;
  hipStream_t st = (hipStream_t)stream;
  jf_status s = check_rows(m, R, st);
  if (s != JF_OK) return s;
  const PackedSpec pk{n_blocks, n, mask};
  SegArgs unused{};
  PROF(JF_KERNEL_STEP);
  s = forward(m, d_tokens, R, unused, 1, d_argmax, d_logits, st, &pk);
  if (s != JF_OK) return s;
  PROF(JF_KERNEL_STEP);
  m->last_rows = 0;  // nothing to commit: the packed rows are not a draft
  return JF_OK;
}

extern "C" jf_status jf_commit_kv(jf_model* m, const int32_t* d_path, const jf_step_result* d_result,
                                  int32_t max_commit, jf_stream stream) {
  if (!m || !d_result) return fail(JF_E_INVAL, "null pointer argument");
  if (m->last_rows == 0) return fail(JF_E_STATE, "no step to commit");
  if (m->last_tree && !d_path) return fail(JF_E_INVAL, "a multi-block step needs its path");
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(launch_commit(m->cfg.dtype, m->kv, m->cfg.n_layers, m->L.n_pages, m->cfg.n_kv_heads,
                        m->cfg.head_dim, m->at<int32_t>(m->L.w_pt), m->state(), d_path,
                        reinterpret_cast<const int32_t*>(d_result), max_commit, 0, m->cfg.max_ctx, st));
  int add = m->last_rows;
  if (max_commit > 0 && max_commit < add) add = max_commit;
  m->C_ub = std::min(m->C_ub + add, m->cfg.max_ctx);
  m->last_rows = 0;
  return JF_OK;
}

extern "C" jf_status jf_kv_length(jf_model* m, int32_t* out, jf_stream stream) {
  if (!m || !out) return fail(JF_E_INVAL, "null pointer argument");
  hipStream_t st = (hipStream_t)stream;
  int32_t v = 0;
  HIP_TRY(hipMemcpyAsync(&v, m->state(), 4, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  *out = v;
  m->C_ub = v;
  return JF_OK;
}

extern "C" jf_status jf_kv_truncate(jf_model* m, int32_t new_len, jf_stream stream) {
  if (!m) return fail(JF_E_INVAL, "model is null");
  int32_t C = 0;
  jf_status s = jf_kv_length(m, &C, stream);
  if (s != JF_OK) return s;
  if (new_len < 0 || new_len > C) return fail(JF_E_STATE, "truncate to %d, committed length is %d", new_len, C);
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(launch_set_int(m->state(), new_len, st));
  HIP_TRY(hipStreamSynchronize(st));
  m->C_ub = new_len;
  m->last_rows = 0;
  return JF_OK;
}

extern "C" jf_status jf_kv_set_page_table(jf_model* m, const int32_t* h_table, int32_t n, jf_stream stream) {
  if (!m || !h_table) return fail(JF_E_INVAL, "null pointer argument");
  if (n != m->L.n_pages) return fail(JF_E_INVAL, "page table needs %d entries, got %d", m->L.n_pages, n);
  std::vector<char> seen(n, 0);
  for (int i = 0; i < n; ++i) {
    if (h_table[i] < 0 || h_table[i] >= n || seen[h_table[i]])
      return fail(JF_E_INVAL, "page table entry %d is out of range or repeated", i);
    seen[h_table[i]] = 1;
  }
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(hipMemcpyAsync(m->ws + m->L.w_pt, h_table, (size_t)n * 4, hipMemcpyHostToDevice, st));
  HIP_TRY(hipStreamSynchronize(st));
  return JF_OK;
}

// ---- component calls ---------------------------------------------------------------------
extern "C" size_t jf_attention_ws_bytes(int32_t n_heads, int32_t head_dim, int32_t R) {
  if (n_heads < 1 || head_dim < 1 || R < 1) return 0;
  // split partials: o, then (max, sum)
  return (size_t)kAttnMaxSplits * R * n_heads * (head_dim + 2) * 4 + 256;
}

extern "C" jf_status jf_attention(int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, int32_t dtype,
                                  int32_t C, int32_t R, const void* d_q, const void* d_kv_layer,
                                  const int32_t* d_page_table, const uint64_t* d_vis, void* d_out,
                                  void* d_ws, jf_stream stream) {
  if (!d_q || !d_kv_layer || !d_page_table || !d_out || !d_ws) return fail(JF_E_INVAL, "null pointer argument");
  if (dtype != JF_F32 && dtype != JF_BF16) return fail(JF_E_DTYPE, "dtype %d unsupported", dtype);
  if (n_heads < 1 || n_kv_heads < 1 || n_heads % n_kv_heads) return fail(JF_E_SHAPE, "bad head counts");
  if (head_dim != 32 && head_dim != 64 && head_dim != 128) return fail(JF_E_SHAPE, "head_dim must be 32, 64 or 128");
  if (R < 1 || R > kMaxRows || C < 0) return fail(JF_E_CAPACITY, "R must be in [1, %d] and C >= 0", kMaxRows);
  AttnArgs a{};
  a.H = n_heads; a.G = n_kv_heads; a.hd = head_dim; a.R = R; a.max_ctx = C + R;
  a.keys_ub = C + R;
  a.lds_ok = dtype == JF_BF16;
  attn_plan(a);
  a.q = d_q; a.q_plane = (size_t)R * n_heads * head_dim;
  a.kv = d_kv_layer; a.page_table = d_page_table; a.state = nullptr; a.C_host = C;
  a.vis = d_vis;
  a.out_plane = (size_t)(R + 15) / 16 * 16 * n_heads * head_dim;  // GEMM-input layout, rows padded to 16
  a.o_part = (float*)d_ws;
  a.ml_part = (float*)((char*)d_ws + (size_t)kAttnMaxSplits * R * n_heads * head_dim * 4);
  a.out = d_out;
  HIP_TRY(launch_attention(dtype, a, (hipStream_t)stream));
  return JF_OK;
}

extern "C" size_t jf_packed_matrix_bytes(int32_t rows, int32_t cols, int32_t dtype) {
  if (rows < 1 || cols < 1) return 0;
  return (size_t)rows * cols * (dtype == JF_BF16 ? 2 : 4);
}

extern "C" jf_status jf_pack_matrix(int32_t rows, int32_t cols, int32_t dtype, const void* d_src,
                                    void* d_packed, jf_stream stream) {
  if (!d_src || !d_packed) return fail(JF_E_INVAL, "null pointer argument");
  if (dtype != JF_F32 && dtype != JF_BF16) return fail(JF_E_DTYPE, "dtype %d unsupported", dtype);
  if (rows < 16 || rows % 16 || cols < 128 || cols % 128)
    return fail(JF_E_SHAPE, "rows must be a multiple of 16 and cols of 128");
  const void* src[1] = {d_src};
  HIP_TRY(launch_pack(dtype, rows, cols, src, 1, nullptr, d_packed, (hipStream_t)stream));
  return JF_OK;
}

extern "C" size_t jf_lm_head_ws_bytes(int32_t R, int32_t V) {
  if (R < 1 || V < 16) return 0;
  return (size_t)(V / 16) * R * 8 + 256;
}

extern "C" jf_status jf_lm_head_accept(int32_t R, int32_t d, int32_t V, int32_t dtype, const void* d_x,
                                       const void* d_w_packed, const int32_t* d_draft, int32_t* d_argmax,
                                       jf_step_result* d_result, float* d_logits, void* d_ws,
                                       jf_stream stream) {
  if (!d_x || !d_w_packed || !d_argmax || !d_ws) return fail(JF_E_INVAL, "null pointer argument");
  if (d_draft && !d_result) return fail(JF_E_INVAL, "acceptance needs d_result");
  if (dtype != JF_F32 && dtype != JF_BF16) return fail(JF_E_DTYPE, "dtype %d unsupported", dtype);
  if (R < 1 || R > kMaxRows) return fail(JF_E_CAPACITY, "R must be in [1, %d]", kMaxRows);
  if (d < 128 || d % 128 || V < 16 || V % 16) return fail(JF_E_SHAPE, "d multiple of 128, V multiple of 16");
  hipStream_t st = (hipStream_t)stream;
  Epi ep{};
  ep.kind = EPI_ARGMAX; ep.R = R; ep.part = (uint64_t*)d_ws; ep.part_stride = R;
  ep.logits = d_logits; ep.ldl = V;
  int part_blocks = 0;
  // no split-K scratch in the component call
  HIP_TRY(run_gemm(dtype, R, V, d, d_x, (size_t)(R + 15) / 16 * 16 * d, d_w_packed, ep, st, &part_blocks, false));
  HIP_TRY(launch_argmax_reduce(ep.part, part_blocks, R, R, d_argmax, st));
  if (d_draft) {
    int32_t* zero = (int32_t*)((char*)d_ws + (size_t)(V / 16) * R * 8);
    HIP_TRY(launch_set_int(zero, 0, st));
    HIP_TRY(launch_accept_linear(d_draft, d_argmax, R, 0, 0, V, zero, nullptr,
                                 reinterpret_cast<int32_t*>(d_result), nullptr, st));
  }
  return JF_OK;
}

// ---- the LM-head component without caller workspace ----------------------------------
// Its scratch (the per-block argmax keys and the zeroed committed-length word
// the acceptance kernel takes) lives in this fixed device array: one copy per
// GPU, held until the process ends.  Host code never passes the array's name
// to a kernel (in host code it is a stand-in, not a device address); it uses
// the device address read once per device with hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[JF_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// Device address of `scratch` on the current device (looked up once per device).
static jf_status scratch_ptr(void** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(JF_E_INVAL, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(JF_E_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return JF_OK;
}

extern "C" jf_status jf_lm_head_accept_noalloc(int32_t R, int32_t d, int32_t V, int32_t dtype, const void* d_x,
                                               const void* d_w_packed, const int32_t* d_draft, int32_t* d_argmax,
                                               jf_step_result* d_result, float* d_logits, jf_stream stream) {
  if (!d_x || !d_w_packed || !d_argmax) return fail(JF_E_INVAL, "null pointer argument");
  if (d_draft && !d_result) return fail(JF_E_INVAL, "acceptance needs d_result");
  if (dtype != JF_F32 && dtype != JF_BF16) return fail(JF_E_DTYPE, "dtype %d unsupported", dtype);
  if (R < 1 || R > kMaxRows) return fail(JF_E_CAPACITY, "R must be in [1, %d]", kMaxRows);
  if (d < 128 || d % 128 || V < 16 || V % 16) return fail(JF_E_SHAPE, "d multiple of 128, V multiple of 16");
  const size_t need = jf_lm_head_ws_bytes(R, V);
  if (need > JF_NOALLOC_SCRATCH_BYTES)
    return fail(JF_E_CAPACITY, "R = %d, V = %d need %zu bytes of scratch; the fixed scratch holds %zu", R, V, need,
                (size_t)JF_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  jf_status s = scratch_ptr(&ws);
  if (s != JF_OK) return s;
  return jf_lm_head_accept(R, d, V, dtype, d_x, d_w_packed, d_draft, d_argmax, d_result, d_logits, ws, stream);
}

// ---- trajectories ------------------------------------------------------------------------
extern "C" jf_status jf_trajectory_record(const int32_t* d_prev, const int32_t* d_argmax, int32_t n,
                                          int32_t rows, int32_t* d_out, jf_stream stream) {
  if (!d_prev || !d_argmax || !d_out) return fail(JF_E_INVAL, "null pointer argument");
  if (n < 1 || rows < 1 || rows > n) return fail(JF_E_SHAPE, "need 1 <= rows <= n (n = %d, rows = %d)", n, rows);
  HIP_TRY(launch_traj_record(d_prev, d_argmax, n, rows, d_out, (hipStream_t)stream));
  return JF_OK;
}

extern "C" jf_status jf_trajectory_select(const int32_t* d_traj, const int32_t* d_len, int32_t n_blocks,
                                          int32_t n, int32_t max_points, int32_t w, const int32_t* d_t_num,
                                          int32_t* d_sel, int32_t* d_unconv, jf_stream stream) {
  if (!d_traj || !d_len || !d_sel) return fail(JF_E_INVAL, "null pointer argument");
  if (n_blocks < 0 || n < 1 || max_points < 1 || w < 1)
    return fail(JF_E_SHAPE, "need n_blocks >= 0 and n, max_points, w >= 1");
  if (n_blocks == 0) return JF_OK;
  HIP_TRY(launch_traj_select(d_traj, d_len, n_blocks, n, max_points, w, d_t_num, d_sel, d_unconv,
                             (hipStream_t)stream));
  return JF_OK;
}
