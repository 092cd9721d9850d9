// Host side of libmarche.so: argument validation, workspace layout, the
// per-layer launch sequence of a cache-aware decoder step, error reporting
// and optional per-kernel timing.  Public contract: include/marche.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include <cstdlib>

#include "../../include/marche.h"
#include "marche_host.h"
#include "marche_internal.h"

using namespace marche;

int marche::device_cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64) {
    const int v = cached[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  if (dev < 64) cached[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

namespace {

thread_local std::string t_err;

// Debug mode: MARCHE_VALIDATE set to anything but "" or "0" makes every step
// check its device-resident active lists before launching (read per call).
bool validate_requested() {
  const char *v = std::getenv("MARCHE_VALIDATE");
  return v && v[0] && !(v[0] == '0' && v[1] == 0);
}

marche_status_t fail(marche_status_t s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  t_err = buf;
  return s;
}

marche_status_t fail_hip(hipError_t e, const char *what) {
  return fail(MARCHE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// The int a caller stored in an enum-typed field or argument.  A C caller may
// store any int there, and in C++ reading an enum object whose value lies
// outside the enumeration's range is undefined, so caller-supplied enums are
// read through their object representation before they are validated.
template <class E>
int32_t raw_enum(const E &e) {
  static_assert(sizeof(E) == sizeof(int32_t), "C enums are int-sized");
  int32_t v;
  std::memcpy(&v, &e, sizeof v);
  return v;
}

size_t elem_size(int32_t dt) { return dt == MARCHE_BF16 ? 2 : 4; }

marche_status_t check_model(const marche_model_t *m) {
  if (!m) return fail(MARCHE_ERR_INVALID_ARG, "model is NULL");
  if (m->n_layers < 1) return fail(MARCHE_ERR_INVALID_ARG, "model.n_layers=%d < 1", m->n_layers);
  if (m->n_heads < 1 || m->head_dim < 1 || m->d_model != m->n_heads * m->head_dim)
    return fail(MARCHE_ERR_INVALID_ARG, "model.d_model=%d != n_heads*head_dim (%d*%d)", m->d_model,
                m->n_heads, m->head_dim);
  if (raw_enum(m->dtype) != MARCHE_F32 && raw_enum(m->dtype) != MARCHE_BF16)
    return fail(MARCHE_ERR_UNSUPPORTED, "model.dtype=%d is not F32 or BF16", raw_enum(m->dtype));
  if (m->head_dim != 64 && m->head_dim != 80)
    return fail(MARCHE_ERR_UNSUPPORTED, "model.head_dim=%d (supported: 64, 80)", m->head_dim);
  if (m->d_model % 256 != 0 || m->d_model > 2048)
    return fail(MARCHE_ERR_UNSUPPORTED, "model.d_model=%d (must be a multiple of 256, <= 2048)",
                m->d_model);
  if (m->d_mlp < 256 || m->d_mlp % 256 != 0)
    return fail(MARCHE_ERR_UNSUPPORTED, "model.d_mlp=%d (must be a positive multiple of 256)",
                m->d_mlp);
  if (m->n_tokens < 1 || m->n_tokens > 4096)
    return fail(MARCHE_ERR_INVALID_ARG, "model.n_tokens=%d (must be in [1, 4096])", m->n_tokens);
  if (!(m->ln_eps > 0.0f)) return fail(MARCHE_ERR_INVALID_ARG, "model.ln_eps must be > 0");
  return MARCHE_OK;
}

// ------------------------------------------------------------------ profiling

// One class per kernel symbol.  The attention kernel is instantiated per
// query-chunk width (1, 2, 4 or 8 wavefronts of 32 queries), chosen from the
// largest active set of the call; each bf16 GEMM has a 128x256, a 256x256
// (class + 1), a 64x128 (_S), a 128x128 (_M) and a 320x256 (_I) tile
// instantiation, chosen from its shape (fp32 GEMMs are timed under the
// first).
enum KClass {
  K_ROW_MAP, K_GATHER_LN, K_GEMM_QKV, K_GEMM_QKV_L, K_ATTN_W1, K_ATTN_W2, K_ATTN_W4,
  K_ATTN_SCORES, K_GEMM_O, K_GEMM_O_L, K_GEMM_FC1, K_GEMM_FC1_L, K_GEMM_FC2, K_GEMM_FC2_L,
  K_SELECT, K_DECODER_INPUT, K_FILL, K_ATTN2_W1, K_ATTN2_W2, K_ATTN2_W4, K_CONCAT, K_ATTN_RES,
  K_ENC_INPUT, K_MASK_FILL, K_LN_ROWS, K_GEMM_EMBED, K_GEMM_EMBED_L, K_TIME_SINUS, K_GEMM_HEAD,
  K_GEMM_HEAD_L, K_GEMM_HEAD_SILU, K_GEMM_HEAD_SILU_L, K_HEAD_SILU_COND, K_HEAD_IN_MOD,
  K_HEAD_GATE_MOD, K_HEAD_OUT_STEP, K_GEMM_QKV_S, K_GEMM_O_S, K_GEMM_FC1_S, K_GEMM_FC2_S,
  K_GEMM_EMBED_S, K_GEMM_HEAD_S, K_GEMM_HEAD_SILU_S, K_TRANSPOSE, K_GEMM_QKV_M, K_GEMM_O_M,
  K_GEMM_FC1_M, K_GEMM_FC2_M, K_GEMM_EMBED_M, K_GEMM_HEAD_M, K_GEMM_HEAD_SILU_M,
  K_ATTN_RES_SC, K_ATTN_W8, K_ATTN_SC, K_GEMM_QKV_I, K_GEMM_O_I, K_GEMM_FC1_I, K_GEMM_FC2_I,
  K_GEMM_EMBED_I, K_GEMM_HEAD_I, K_GEMM_HEAD_SILU_I,
  K_NCLASS
};
const char *const kClassNames[K_NCLASS] = {
    "row_map",           "gather_ln",      "gemm_qkv_t128x256", "gemm_qkv_t256",
    "attention_q32",     "attention_q64",  "attention_q128",    "attn_scores",
    "gemm_o_t128x256",   "gemm_o_t256",    "gemm_fc1_t128x256", "gemm_fc1_t256",
    "gemm_fc2_t128x256", "gemm_fc2_t256",  "select_topk",       "decoder_input",
    "fill_zero",         "attention2_q32", "attention2_q64",    "attention2_q128",
    "concat_kv",         "attention_res",  "encoder_input",     "mask_fill",
    "ln_rows",           "gemm_embed_t128x256", "gemm_embed_t256", "time_sinus",
    "gemm_head_t128x256", "gemm_head_t256", "gemm_head_silu_t128x256", "gemm_head_silu_t256",
    "head_silu_cond",    "head_in_mod",    "head_gate_mod",     "head_out_step",
    "gemm_qkv_t64x128",  "gemm_o_t64x128", "gemm_fc1_t64x128",  "gemm_fc2_t64x128",
    "gemm_embed_t64x128", "gemm_head_t64x128", "gemm_head_silu_t64x128", "transpose",
    "gemm_qkv_t128",     "gemm_o_t128",    "gemm_fc1_t128",     "gemm_fc2_t128",
    "gemm_embed_t128",   "gemm_head_t128", "gemm_head_silu_t128", "attention_res_scores", "attention_q256",
    "attention_scores",  "gemm_qkv_t320",  "gemm_o_t320",      "gemm_fc1_t320",
    "gemm_fc2_t320",     "gemm_embed_t320", "gemm_head_t320",  "gemm_head_silu_t320"};
static_assert(sizeof(kClassNames) / sizeof(kClassNames[0]) == K_NCLASS, "one name per class");

// Launches inside marche_step in layers where not every token of every image
// is active (cache-aware layers) are timed under a class of their own: the
// class index + K_NCLASS, named with the suffix "_ca".  A class without the
// suffix then holds only full-layer launches (or launches outside the step),
// whose hardware counters a one-step run at a full step measures.
constexpr int K_NTIMED = 2 * K_NCLASS;

const char *class_name(int i) {
  static const std::vector<std::string> names = [] {
    std::vector<std::string> v;
    for (int j = 0; j < K_NCLASS; ++j) v.emplace_back(kClassNames[j]);
    for (int j = 0; j < K_NCLASS; ++j) v.emplace_back(std::string(kClassNames[j]) + "_ca");
    return v;
  }();
  return names[i].c_str();
}

// Timing class of a GEMM launch: base is the projection's 128x256 class, the
// 256x256 class follows it; the 64x128 classes are listed separately.
int gemm_class(int base, DType dt, int32_t m, int32_t n, int32_t k) {
  const int kind = gemm_tile_kind(dt, m, n, k);
  if (kind == GEMM_TILE_256) return base + 1;
  if (kind == GEMM_TILE_320) {
    switch (base) {
      case K_GEMM_QKV: return K_GEMM_QKV_I;
      case K_GEMM_O: return K_GEMM_O_I;
      case K_GEMM_FC1: return K_GEMM_FC1_I;
      case K_GEMM_FC2: return K_GEMM_FC2_I;
      case K_GEMM_EMBED: return K_GEMM_EMBED_I;
      case K_GEMM_HEAD: return K_GEMM_HEAD_I;
      default: return K_GEMM_HEAD_SILU_I;
    }
  }
  if (kind == GEMM_TILE_128) {
    switch (base) {
      case K_GEMM_QKV: return K_GEMM_QKV_M;
      case K_GEMM_O: return K_GEMM_O_M;
      case K_GEMM_FC1: return K_GEMM_FC1_M;
      case K_GEMM_FC2: return K_GEMM_FC2_M;
      case K_GEMM_EMBED: return K_GEMM_EMBED_M;
      case K_GEMM_HEAD: return K_GEMM_HEAD_M;
      default: return K_GEMM_HEAD_SILU_M;
    }
  }
  if (kind != GEMM_TILE_64x128) return base;
  switch (base) {
    case K_GEMM_QKV: return K_GEMM_QKV_S;
    case K_GEMM_O: return K_GEMM_O_S;
    case K_GEMM_FC1: return K_GEMM_FC1_S;
    case K_GEMM_FC2: return K_GEMM_FC2_S;
    case K_GEMM_EMBED: return K_GEMM_EMBED_S;
    case K_GEMM_HEAD: return K_GEMM_HEAD_S;
    default: return K_GEMM_HEAD_SILU_S;
  }
}

int attn_class(DType dt, int a_max, int n_tokens, int head_dim) {
  if (dt == DType::BF16 && attn_resident(a_max, n_tokens, false)) return K_ATTN_RES;
  if (a_max > 128 && dt == DType::BF16 && attn_streams(head_dim, n_tokens, false)) return K_ATTN_W8;
  return a_max <= 32 ? K_ATTN_W1 : (a_max <= 64 ? K_ATTN_W2 : K_ATTN_W4);
}

struct Pending {
  int cls;
  hipEvent_t e0, e1;
  double flops, bytes;
};
struct Totals {
  int64_t launches = 0;
  double ms = 0, flops = 0, bytes = 0;
};

std::mutex g_mu;
bool g_prof = false;
thread_local KernelEvents *t_kernel_events = nullptr;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
Totals g_tot[K_NTIMED];

hipEvent_t pool_get() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Times one launch call when profiling is on: its first kernel's dispatch
// carries the two events (launch_kernel), so they hold that kernel's own
// start and end.  A call that launches no kernel records nothing.
struct ProfScope {
  int cls;
  double flops, bytes;
  KernelEvents ev;
  bool on = false;
  ProfScope(int c, double f, double b) : cls(c), flops(f), bytes(b) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_prof) return;
    ev.start = pool_get();
    ev.stop = pool_get();
    if (!ev.start || !ev.stop) return;
    on = true;
    kernel_events() = &ev;
  }
  void done() {
    if (!on) return;
    kernel_events() = nullptr;
    std::lock_guard<std::mutex> lk(g_mu);
    if (ev.used) {
      g_pending.push_back({cls, ev.start, ev.stop, flops, bytes});
    } else {
      g_pool.push_back(ev.start);
      g_pool.push_back(ev.stop);
    }
    on = false;
  }
  ~ProfScope() {
    if (on) kernel_events() = nullptr;
  }
};

#define LAUNCH(cls, flops, bytes, call)                        \
  do {                                                         \
    ProfScope ps_(cls, (double)(flops), (double)(bytes));      \
    hipError_t e_ = (call);                                    \
    ps_.done();                                                \
    if (e_ != hipSuccess) return fail_hip(e_, #call);          \
  } while (0)

}  // namespace

marche::KernelEvents *&marche::kernel_events() { return t_kernel_events; }

marche_status_t marche::set_error(marche_status_t s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  t_err = buf;
  return s;
}

// ------------------------------------------------------------------ ABI

extern "C" {

const char *marche_status_string(marche_status_t s) {
  switch (raw_enum(s)) {
    case MARCHE_OK: return "MARCHE_OK";
    case MARCHE_ERR_INVALID_ARG: return "MARCHE_ERR_INVALID_ARG";
    case MARCHE_ERR_UNSUPPORTED: return "MARCHE_ERR_UNSUPPORTED";
    case MARCHE_ERR_HIP: return "MARCHE_ERR_HIP";
    case MARCHE_ERR_WORKSPACE: return "MARCHE_ERR_WORKSPACE";
  }
  return "MARCHE_STATUS_UNKNOWN";
}

const char *marche_last_error(void) { return t_err.c_str(); }

marche_status_t kv_cache_init(marche_kv_cache_t *cache, const marche_model_t *m, int32_t batch,
                              void *k_buf, void *v_buf, size_t bytes_each, const void *k_init,
                              const void *v_init, marche_stream_t stream_) {
  if (!cache) return fail(MARCHE_ERR_INVALID_ARG, "cache is NULL");
  marche_status_t st = check_model(m);
  if (st != MARCHE_OK) return st;
  if (batch < 0) return fail(MARCHE_ERR_INVALID_ARG, "batch=%d < 0", batch);
  if (!k_buf || !v_buf) return fail(MARCHE_ERR_INVALID_ARG, "k_buf / v_buf is NULL");
  if ((k_init == nullptr) != (v_init == nullptr))
    return fail(MARCHE_ERR_INVALID_ARG, "k_init and v_init must both be given or both be NULL");
  const size_t need = (size_t)m->n_layers * batch * m->n_heads * m->n_tokens * m->head_dim *
                      elem_size(m->dtype);
  if (bytes_each < need)
    return fail(MARCHE_ERR_INVALID_ARG, "bytes_each=%zu < %zu needed", bytes_each, need);
  if ((reinterpret_cast<uintptr_t>(k_buf) | reinterpret_cast<uintptr_t>(v_buf)) & 15)
    return fail(MARCHE_ERR_INVALID_ARG, "k_buf / v_buf must be 16-byte aligned");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  cache->k = k_buf;
  cache->v = v_buf;
  cache->n_layers = m->n_layers;
  cache->batch = batch;
  cache->n_heads = m->n_heads;
  cache->n_tokens = m->n_tokens;
  cache->head_dim = m->head_dim;
  cache->dtype = m->dtype;
  if (need == 0) return MARCHE_OK;
  if (k_init) {
    hipError_t e = hipMemcpyAsync(k_buf, k_init, need, hipMemcpyDeviceToDevice, stream);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpyAsync(k_init)");
    e = hipMemcpyAsync(v_buf, v_init, need, hipMemcpyDeviceToDevice, stream);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpyAsync(v_init)");
    return MARCHE_OK;
  }
  LAUNCH(K_FILL, 0, need, launch_fill_zero(k_buf, need, stream));
  LAUNCH(K_FILL, 0, need, launch_fill_zero(v_buf, need, stream));
  return MARCHE_OK;
}

size_t marche_step_workspace_bytes(const marche_model_t *m, int32_t batch, int32_t a_total) {
  (void)batch;
  if (!m || a_total < 0) return 0;
  const size_t es = elem_size(raw_enum(m->dtype));
  const size_t M = (size_t)a_total;
  return align256(M * sizeof(RowMap)) + 2 * align256(M * m->d_model * es) +
         align256(M * m->d_mlp * es);
}

}  // extern "C"

marche_status_t marche::step_impl(const marche_model_t *m, const marche_layer_t *layers,
                                  const marche_kv_cache_t *cache, int32_t first_image,
                                  int32_t layer_begin, int32_t layer_end, int32_t batch, float *x,
                                  const int32_t *a_idx, const int32_t *a_off, const int32_t *n_gen,
                                  int32_t a_total, int32_t a_max, int32_t gen_max, float *scores,
                                  int32_t score_layer, void *workspace, size_t workspace_bytes,
                                  marche_stream_t stream_) {
  marche_status_t st = check_model(m);
  if (st != MARCHE_OK) return st;
  if (!layers) return fail(MARCHE_ERR_INVALID_ARG, "layers is NULL");
  if (!cache || !cache->k || !cache->v) return fail(MARCHE_ERR_INVALID_ARG, "cache is NULL or unbound");
  if (cache->n_layers != m->n_layers || cache->n_heads != m->n_heads ||
      cache->n_tokens != m->n_tokens || cache->head_dim != m->head_dim ||
      raw_enum(cache->dtype) != raw_enum(m->dtype))
    return fail(MARCHE_ERR_INVALID_ARG, "cache shape/dtype does not match the model");
  if (batch < 0 || batch > cache->batch)
    return fail(MARCHE_ERR_INVALID_ARG, "batch=%d outside [0, cache.batch=%d]", batch, cache->batch);
  if (first_image < 0 || first_image > cache->batch - batch)
    return fail(MARCHE_ERR_INVALID_ARG, "images [%d, %d) outside the cache's [0, %d)", first_image,
                first_image + batch, cache->batch);
  if (layer_begin < 0 || layer_end < layer_begin || layer_end > m->n_layers)
    return fail(MARCHE_ERR_INVALID_ARG, "layer range [%d, %d) outside [0, %d]", layer_begin,
                layer_end, m->n_layers);
  if (a_total < 0 || a_total > batch * m->n_tokens)
    return fail(MARCHE_ERR_INVALID_ARG, "a_total=%d outside [0, batch*n_tokens=%d]", a_total,
                batch * m->n_tokens);
  if (a_max < 0 || a_max > m->n_tokens || a_max > a_total || (a_total > 0 && a_max == 0))
    return fail(MARCHE_ERR_INVALID_ARG, "a_max=%d inconsistent with a_total=%d, n_tokens=%d",
                a_max, a_total, m->n_tokens);
  if (gen_max < 0 || gen_max > a_max)
    return fail(MARCHE_ERR_INVALID_ARG, "gen_max=%d outside [0, a_max=%d]", gen_max, a_max);
  {
    // GEMM epilogues address x, the KV slice of a layer and the packed
    // activations with 32-bit element offsets
    const int64_t widest = std::max<int64_t>(3LL * m->d_model, m->d_mlp);
    if ((int64_t)batch * m->n_tokens * m->d_model >= (1LL << 31) ||
        (int64_t)a_total * widest >= (1LL << 31))
      return fail(MARCHE_ERR_UNSUPPORTED,
                  "batch*n_tokens*d_model or a_total*max(3*d_model, d_mlp) reaches 2^31 elements");
  }
  if (layer_begin == layer_end || batch == 0 || a_total == 0) return MARCHE_OK;
  if (!x) return fail(MARCHE_ERR_INVALID_ARG, "x is NULL");
  if (!a_idx || !a_off) return fail(MARCHE_ERR_INVALID_ARG, "a_idx / a_off is NULL");
  const bool want_scores = scores && score_layer >= layer_begin && score_layer < layer_end;
  if (want_scores && !n_gen) return fail(MARCHE_ERR_INVALID_ARG, "scores requested but n_gen is NULL");
  for (int l = layer_begin; l < layer_end; ++l) {
    const marche_layer_t &L = layers[l];
    if (!L.ln1_g || !L.ln1_b || !L.w_qkv || !L.b_qkv || !L.w_o || !L.b_o || !L.ln2_g ||
        !L.ln2_b || !L.w_1 || !L.b_1 || !L.w_2 || !L.b_2)
      return fail(MARCHE_ERR_INVALID_ARG, "layers[%d] has a NULL parameter", l);
  }
  const size_t need = marche_step_workspace_bytes(m, batch, a_total);
  if (!workspace || workspace_bytes < need)
    return fail(MARCHE_ERR_WORKSPACE, "workspace %s: %zu bytes < %zu needed",
                workspace ? "too small" : "is NULL", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) & 255)
    return fail(MARCHE_ERR_INVALID_ARG, "workspace must be 256-byte aligned");

  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (validate_requested()) {
    // the first word of the workspace (the row map's, rewritten below)
    int32_t *report = static_cast<int32_t *>(workspace);
    hipError_t e = launch_check_active(a_idx, a_off, n_gen, batch, m->n_tokens, a_total, a_max,
                                       gen_max, report, stream);
    int32_t h = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(&h, report, sizeof h, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return fail_hip(e, "active-list validation");
    if (h != 0) {
      static const char *what[] = {"a_off inconsistent with a_total / a_max",
                                   "token outside [0, n_tokens)", "token listed twice",
                                   "n_gen outside [0, |A_b|] or above gen_max"};
      const int code = (h - 1) / batch, image = (h - 1) % batch;
      return fail(MARCHE_ERR_INVALID_ARG, "active lists: %s (image %d of the call)",
                  what[code & 3], image);
    }
  }
  const DType dt = m->dtype == MARCHE_BF16 ? DType::BF16 : DType::F32;
  const size_t es = elem_size(m->dtype);
  const int D = m->d_model, F = m->d_mlp, H = m->n_heads, dh = m->head_dim, N = m->n_tokens;
  const int M = a_total;

  char *ws = static_cast<char *>(workspace);
  RowMap *map = reinterpret_cast<RowMap *>(ws);
  ws += align256((size_t)M * sizeof(RowMap));
  void *buf0 = ws;  // LN1 output, then attention output
  ws += align256((size_t)M * D * es);
  void *buf1 = ws;  // queries, then LN2 output
  ws += align256((size_t)M * D * es);
  void *hid = ws;   // MLP hidden activations

  const size_t layer_elems = (size_t)cache->batch * H * N * dh;
  const double gemm_bytes_act = (double)es;

  // timing class offset: cache-aware layers (not every token active) apart
  const int ko = (int64_t)a_total == (int64_t)batch * N ? 0 : K_NCLASS;
  LAUNCH(K_ROW_MAP + ko, 0, (double)M * (4 + sizeof(RowMap)),
         launch_row_map(map, a_idx, a_off, batch, N, stream));

  for (int l = layer_begin; l < layer_end; ++l) {
    const marche_layer_t &L = layers[l];
    // layer l, image first_image: the call's image 0
    const size_t base = ((size_t)l * layer_elems + (size_t)first_image * H * N * dh) * es;
    char *kc = static_cast<char *>(cache->k) + base;
    char *vc = static_cast<char *>(cache->v) + base;

    LAUNCH(K_GATHER_LN + ko, 0, (double)M * D * (4 + es),
           launch_gather_ln(dt, buf0, x, map, static_cast<const float *>(L.ln1_g),
                            static_cast<const float *>(L.ln1_b), M, D, m->ln_eps, stream));
    QkvOut qo{buf1, kc, vc, D, dh, H, N};
    LAUNCH(gemm_class(K_GEMM_QKV, dt, M, 3 * D, D) + ko, 2.0 * M * 3 * D * D,
           gemm_bytes_act * ((double)M * D + 3.0 * D * D + 3.0 * M * D),
           launch_gemm_qkv(dt, buf0, L.w_qkv, static_cast<const float *>(L.b_qkv), M, 3 * D, D,
                           map, qo, stream));
    AttnArgs aa{buf1, kc, vc, buf0, a_off, map, batch, H, N, dh, D, M, a_max};
    // At the selection layer the resident attention kernel also writes the
    // score pass (Section 4.2) from the K tiles it holds; other sizes run the
    // score pass as a kernel of its own after the attention.
    const bool sel = want_scores && l == score_layer;
    const bool fused = sel && dt == DType::BF16 && attn_fuses_scores(a_max, N, dh, gen_max);
    if (fused) {
      aa.n_gen = n_gen;
      aa.scores = scores;
    }
    // Algorithmic traffic: every cached K/V element of the batch read once,
    // plus the queries read and the outputs written (and the scores).
    const int acls = attn_class(dt, a_max, N, dh);
    LAUNCH((fused ? (acls == K_ATTN_RES ? K_ATTN_RES_SC : K_ATTN_SC) : acls) + ko,
           4.0 * M * N * D + (fused ? 2.0 * batch * gen_max * N * D : 0.0),
           es * (2.0 * batch * N * D + 2.0 * M * D) + (fused ? 4.0 * batch * H * N : 0.0),
           launch_attention(dt, aa, stream));
    aa.n_gen = nullptr;
    aa.scores = nullptr;
    if (sel && !fused) {
      LAUNCH(K_ATTN_SCORES + ko, 2.0 * batch * gen_max * N * D,
             es * (double)batch * N * D + 4.0 * batch * H * N,
             launch_attn_scores(dt, aa, n_gen, gen_max, scores, stream));
    }
    LAUNCH(gemm_class(K_GEMM_O, dt, M, D, D) + ko, 2.0 * M * D * D, gemm_bytes_act * ((double)M * D + (double)D * D) + 8.0 * M * D,
           launch_gemm_resid(dt, buf0, L.w_o, static_cast<const float *>(L.b_o), M, D, D, map, x,
                             0, stream));
    LAUNCH(K_GATHER_LN + ko, 0, (double)M * D * (4 + es),
           launch_gather_ln(dt, buf1, x, map, static_cast<const float *>(L.ln2_g),
                            static_cast<const float *>(L.ln2_b), M, D, m->ln_eps, stream));
    LAUNCH(gemm_class(K_GEMM_FC1, dt, M, F, D) + ko, 2.0 * M * F * D,
           gemm_bytes_act * ((double)M * D + (double)F * D + (double)M * F),
           launch_gemm_gelu(dt, buf1, L.w_1, static_cast<const float *>(L.b_1), M, F, D, hid,
                            stream));
    LAUNCH(gemm_class(K_GEMM_FC2, dt, M, D, F) + ko, 2.0 * M * D * F,
           gemm_bytes_act * ((double)M * F + (double)D * F) + 8.0 * M * D,
           launch_gemm_resid(dt, hid, L.w_2, static_cast<const float *>(L.b_2), M, D, F, map, x,
                             1, stream));
  }
  return MARCHE_OK;
}

extern "C" {

marche_status_t marche_step(const marche_model_t *m, const marche_layer_t *layers,
                            const marche_kv_cache_t *cache, int32_t layer_begin,
                            int32_t layer_end, int32_t batch, float *x, const int32_t *a_idx,
                            const int32_t *a_off, const int32_t *n_gen, int32_t a_total,
                            int32_t a_max, int32_t gen_max, float *scores, int32_t score_layer,
                            void *workspace, size_t workspace_bytes, marche_stream_t stream) {
  return step_impl(m, layers, cache, 0, layer_begin, layer_end, batch, x, a_idx, a_off, n_gen,
                   a_total, a_max, gen_max, scores, score_layer, workspace, workspace_bytes, stream);
}

marche_status_t marche_step_images(const marche_model_t *m, const marche_layer_t *layers,
                                   const marche_kv_cache_t *cache, int32_t first_image,
                                   int32_t layer_begin, int32_t layer_end, int32_t batch, float *x,
                                   const int32_t *a_idx, const int32_t *a_off,
                                   const int32_t *n_gen, int32_t a_total, int32_t a_max,
                                   int32_t gen_max, float *scores, int32_t score_layer,
                                   void *workspace, size_t workspace_bytes,
                                   marche_stream_t stream) {
  return step_impl(m, layers, cache, first_image, layer_begin, layer_end, batch, x, a_idx, a_off,
                   n_gen, a_total, a_max, gen_max, scores, score_layer, workspace,
                   workspace_bytes, stream);
}

marche_status_t select_refresh(const float *scores, int32_t n_parts, const int32_t *excl_idx,
                               const int32_t *excl_off, int32_t batch, int32_t n_tokens,
                               int32_t k, int32_t *out_idx, const int32_t *out_off,
                               marche_stream_t stream_) {
  return select_refresh_ordered(scores, n_parts, excl_idx, excl_off, batch, n_tokens, k, out_idx,
                                out_off, MARCHE_SELECT_HIGHEST, stream_);
}

marche_status_t select_refresh_ordered(const float *scores, int32_t n_parts,
                                       const int32_t *excl_idx, const int32_t *excl_off,
                                       int32_t batch, int32_t n_tokens, int32_t k,
                                       int32_t *out_idx, const int32_t *out_off, int32_t order,
                                       marche_stream_t stream_) {
  if (order != MARCHE_SELECT_HIGHEST && order != MARCHE_SELECT_LOWEST)
    return fail(MARCHE_ERR_INVALID_ARG, "order=%d is not HIGHEST or LOWEST", order);
  if (batch < 0) return fail(MARCHE_ERR_INVALID_ARG, "batch=%d < 0", batch);
  if (n_tokens < 1 || n_tokens > 4096)
    return fail(MARCHE_ERR_INVALID_ARG, "n_tokens=%d outside [1, 4096]", n_tokens);
  if (k < 0 || k > n_tokens)
    return fail(MARCHE_ERR_INVALID_ARG, "k=%d outside [0, n_tokens=%d]", k, n_tokens);
  if (n_parts < 1) return fail(MARCHE_ERR_INVALID_ARG, "n_parts=%d < 1", n_parts);
  if (batch == 0 || k == 0) return MARCHE_OK;
  if (!scores || !out_idx || !out_off || !excl_off)
    return fail(MARCHE_ERR_INVALID_ARG, "scores / out_idx / out_off / excl_off is NULL");
  if (!excl_idx) return fail(MARCHE_ERR_INVALID_ARG, "excl_idx is NULL");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  LAUNCH(K_SELECT, 0, 4.0 * batch * n_parts * n_tokens,
         launch_select_topk(scores, n_parts, excl_idx, excl_off, batch, n_tokens, k, out_idx,
                            out_off, order == MARCHE_SELECT_LOWEST, stream));
  return MARCHE_OK;
}

size_t marche_attention_workspace_bytes(int32_t batch, int32_t n_heads, int32_t head_dim,
                                         int32_t n_a, int32_t n_c, int32_t dtype, int32_t mode) {
  if (mode != MARCHE_ATTN_CONCAT || batch <= 0 || n_heads <= 0 || head_dim <= 0 || n_a < 0 ||
      n_c < 0)
    return 0;
  const size_t es = dtype == MARCHE_BF16 ? 2 : 4;
  const size_t one = (size_t)batch * n_heads * (size_t)(n_a + n_c) * head_dim * es;
  return 2 * ((one + 255) & ~(size_t)255);
}

marche_status_t marche_attention_segments(const void *q, void *o, int32_t n_query,
                                          const void *k_a, const void *v_a, int32_t n_a,
                                          const void *k_c, const void *v_c, int32_t n_c,
                                          int32_t batch, int32_t n_heads, int32_t head_dim,
                                          int32_t dtype, int32_t mode, void *workspace,
                                          size_t workspace_bytes, marche_stream_t stream_) {
  if (mode != MARCHE_ATTN_TWO_SEGMENT && mode != MARCHE_ATTN_CONCAT)
    return fail(MARCHE_ERR_INVALID_ARG, "mode=%d is not TWO_SEGMENT or CONCAT", mode);
  if (dtype != MARCHE_BF16)
    return fail(MARCHE_ERR_UNSUPPORTED, "dtype=%d (segment attention is bf16 only)", dtype);
  if (head_dim != 64 && head_dim != 80)
    return fail(MARCHE_ERR_UNSUPPORTED, "head_dim=%d (supported: 64, 80)", head_dim);
  if (batch < 0 || n_heads < 1 || (int64_t)batch * n_heads > 65535)
    return fail(MARCHE_ERR_INVALID_ARG, "batch=%d / n_heads=%d out of range (batch*n_heads <= 65535)",
                batch, n_heads);
  if (n_query < 1 || n_query > 4096)
    return fail(MARCHE_ERR_INVALID_ARG, "n_query=%d outside [1, 4096]", n_query);
  if (n_a < 0 || n_c < 0 || n_a + n_c < 1 || n_a + n_c > 65536)
    return fail(MARCHE_ERR_INVALID_ARG, "segment lengths n_a=%d, n_c=%d (each >= 0, sum in [1, 65536])",
                n_a, n_c);
  const int64_t d_model = (int64_t)n_heads * head_dim;
  if ((int64_t)batch * n_query * d_model >= (1LL << 31) ||
      (int64_t)batch * n_heads * (n_a + n_c) * head_dim >= (1LL << 31))
    return fail(MARCHE_ERR_UNSUPPORTED, "buffers reach 2^31 elements");
  if (batch == 0) return MARCHE_OK;
  if (!q || !o || (n_a > 0 && (!k_a || !v_a)) || (n_c > 0 && (!k_c || !v_c)))
    return fail(MARCHE_ERR_INVALID_ARG, "NULL query, output or non-empty segment");
  for (const void *p : {q, (const void *)o, k_a, v_a, k_c, v_c})
    if (reinterpret_cast<uintptr_t>(p) & 15)
      return fail(MARCHE_ERR_INVALID_ARG, "q, o and the segment buffers must be 16-byte aligned");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  const int cls_w = n_query <= 32 ? 0 : (n_query <= 64 ? 1 : 2);
  const int32_t nt = n_a + n_c;
  const double flops = 4.0 * batch * n_query * (double)nt * d_model;
  // Algorithmic traffic of attention: q, every K/V row of both segments and o once.
  const double attn_bytes =
      2.0 * (2.0 * batch * n_query * d_model + 2.0 * batch * (double)nt * d_model);
  AttnArgs aa{q, k_a, v_a, o, nullptr, nullptr, batch, n_heads, n_a, head_dim,
              (int32_t)d_model, batch * n_query, n_query};
  if (mode == MARCHE_ATTN_TWO_SEGMENT) {
    if (n_a == 0) {  // only the cached segment
      aa.k_cache = k_c;
      aa.v_cache = v_c;
      aa.n_tokens = n_c;
    } else if (n_c > 0) {
      aa.k2 = k_c;
      aa.v2 = v_c;
      aa.n2 = n_c;
    }
    const int cls = (n_a > 0 && n_c > 0) ? K_ATTN2_W1 + cls_w
                                         : attn_class(DType::BF16, n_query, aa.n_tokens, head_dim);
    LAUNCH(cls, flops, attn_bytes, launch_attention(DType::BF16, aa, stream));
    return MARCHE_OK;
  }
  const size_t need =
      marche_attention_workspace_bytes(batch, n_heads, head_dim, n_a, n_c, dtype, mode);
  if (!workspace || workspace_bytes < need)
    return fail(MARCHE_ERR_WORKSPACE, "workspace %s: %zu bytes < %zu needed",
                workspace ? "too small" : "is NULL", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) & 255)
    return fail(MARCHE_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  char *kcat = static_cast<char *>(workspace);
  char *vcat = kcat + need / 2;
  LAUNCH(K_CONCAT, 0, 2.0 * 2.0 * 2.0 * batch * (double)nt * d_model,
         launch_concat_kv(DType::BF16, kcat, vcat, n_a ? k_a : k_c, n_a ? v_a : v_c,
                          n_c ? k_c : k_a, n_c ? v_c : v_a, batch * n_heads, n_a, n_c, head_dim,
                          stream));
  aa.k_cache = kcat;
  aa.v_cache = vcat;
  aa.n_tokens = nt;
  LAUNCH(attn_class(DType::BF16, n_query, nt, head_dim), flops, attn_bytes,
         launch_attention(DType::BF16, aa, stream));
  return MARCHE_OK;
}

marche_status_t marche_decoder_input(float *x, const float *cls, const float *value,
                                     const float *mask, const float *pos, const int32_t *rank,
                                     int32_t batch, int32_t n_tokens, int32_t n_buf,
                                     int32_t d_model, int32_t n_known, marche_stream_t stream_) {
  if (batch < 0 || n_tokens < 1 || n_buf < 0 || n_buf > n_tokens)
    return fail(MARCHE_ERR_INVALID_ARG, "batch=%d n_tokens=%d n_buf=%d inconsistent", batch,
                n_tokens, n_buf);
  if (d_model < 4 || d_model % 4 != 0)
    return fail(MARCHE_ERR_INVALID_ARG, "d_model=%d must be a positive multiple of 4", d_model);
  if (n_known < 0 || n_known > n_tokens - n_buf)
    return fail(MARCHE_ERR_INVALID_ARG, "n_known=%d outside [0, %d]", n_known, n_tokens - n_buf);
  if (batch == 0) return MARCHE_OK;
  if (!x || !cls || !mask || !pos || (n_tokens > n_buf && (!value || !rank)))
    return fail(MARCHE_ERR_INVALID_ARG, "NULL input to marche_decoder_input");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  // Algorithmic traffic: x written once; per-image rows read once (value rows
  // of the tokens generated so far, the class row); the positional rows and the
  // mask row are shared by every image.
  LAUNCH(K_DECODER_INPUT, 0,
         4.0 * d_model * ((double)batch * n_tokens + (double)batch * n_known + batch + n_tokens + 1),
         launch_decoder_input(x, cls, value, mask, pos, rank, batch, n_tokens, n_buf, d_model,
                              n_known, stream));
  return MARCHE_OK;
}

// ------------------------------------------------------------------ rest of a MAR step

marche_status_t marche_encoder_input(float *x_enc, const float *cls, const float *tok,
                                     const float *w_z, const float *b_z, const float *pe_enc,
                                     const int32_t *known, int32_t batch, int32_t n_buf,
                                     int32_t n_img, int32_t n_known, int32_t d_model,
                                     int32_t c_tok, marche_stream_t stream_) {
  if (batch < 0 || n_buf < 0 || n_img < 0 || n_known < 0 || n_known > n_img)
    return fail(MARCHE_ERR_INVALID_ARG, "batch=%d n_buf=%d n_img=%d n_known=%d inconsistent", batch,
                n_buf, n_img, n_known);
  if (d_model < 256 || d_model % 256 != 0 || d_model > 4096)
    return fail(MARCHE_ERR_UNSUPPORTED, "d_model=%d (must be a multiple of 256, <= 4096)", d_model);
  if (c_tok < 1 || c_tok > 64)
    return fail(MARCHE_ERR_UNSUPPORTED, "c_tok=%d (supported: 1..64)", c_tok);
  const int64_t rows = (int64_t)batch * (n_buf + n_known);
  if (rows * d_model >= (1LL << 31)) return fail(MARCHE_ERR_UNSUPPORTED, "x_enc reaches 2^31 elements");
  if (rows == 0) return MARCHE_OK;
  if (!x_enc || !cls || !pe_enc || (n_known > 0 && (!tok || !w_z || !b_z || !known)))
    return fail(MARCHE_ERR_INVALID_ARG, "NULL input to marche_encoder_input");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  // Algorithmic traffic: x_enc written; class, token and positional rows read once.
  LAUNCH(K_ENC_INPUT, 2.0 * batch * n_known * (double)d_model * c_tok,
         4.0 * ((double)rows * d_model + (double)batch * d_model + (double)batch * n_known * c_tok +
                (double)(n_buf + n_img) * d_model + (double)d_model * c_tok),
         launch_encoder_input(x_enc, cls, tok, w_z, b_z, pe_enc, known, batch, n_buf, n_img, n_known,
                              d_model, c_tok, stream));
  return MARCHE_OK;
}

size_t marche_encoder_to_decoder_workspace_bytes(int32_t batch, int32_t n_buf, int32_t n_known,
                                                 int32_t d_model, int32_t dtype) {
  if (batch < 0 || n_buf < 0 || n_known < 0 || d_model < 0) return 0;
  return align256((size_t)batch * (n_buf + n_known) * d_model * elem_size(dtype));
}

marche_status_t marche_encoder_to_decoder(float *x_dec, const float *x_enc, const float *ln_g,
                                          const float *ln_b, float ln_eps, const void *w_de,
                                          const float *b_de, const float *mask,
                                          const float *pe_dec, const int32_t *known,
                                          const int32_t *rank, int32_t batch, int32_t n_buf,
                                          int32_t n_img, int32_t n_known, int32_t d_model,
                                          int32_t dtype, void *workspace, size_t workspace_bytes,
                                          marche_stream_t stream_) {
  if (dtype != MARCHE_F32 && dtype != MARCHE_BF16)
    return fail(MARCHE_ERR_UNSUPPORTED, "dtype=%d is not F32 or BF16", dtype);
  if (batch < 0 || n_buf < 0 || n_img < 0 || n_buf + n_img < 1 || n_known < 0 || n_known > n_img)
    return fail(MARCHE_ERR_INVALID_ARG, "batch=%d n_buf=%d n_img=%d n_known=%d inconsistent", batch,
                n_buf, n_img, n_known);
  if (d_model < 256 || d_model % 256 != 0 || d_model > 4096)
    return fail(MARCHE_ERR_UNSUPPORTED, "d_model=%d (must be a multiple of 256, <= 4096)", d_model);
  if (!(ln_eps > 0.0f)) return fail(MARCHE_ERR_INVALID_ARG, "ln_eps must be > 0");
  const int32_t n_enc = n_buf + n_known, n_tokens = n_buf + n_img;
  // the embedding epilogue addresses x_dec and pe_dec with 32-bit offsets
  if ((int64_t)batch * n_tokens * d_model >= (1LL << 31))
    return fail(MARCHE_ERR_UNSUPPORTED, "x_dec reaches 2^31 elements");
  if (batch == 0) return MARCHE_OK;
  if (!x_dec || !x_enc || !ln_g || !ln_b || !w_de || !b_de || !mask || !pe_dec ||
      (n_img > 0 && !rank) || (n_known > 0 && !known))
    return fail(MARCHE_ERR_INVALID_ARG, "NULL input to marche_encoder_to_decoder");
  const size_t need = marche_encoder_to_decoder_workspace_bytes(batch, n_buf, n_known, d_model, dtype);
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(MARCHE_ERR_WORKSPACE, "workspace %s: %zu bytes < %zu needed",
                workspace ? "too small" : "is NULL", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) & 255)
    return fail(MARCHE_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  const DType dt = dtype == MARCHE_BF16 ? DType::BF16 : DType::F32;
  const size_t es = elem_size(dtype);
  const int M = batch * n_enc, D = d_model;
  if (M > 0) {
    LAUNCH(K_LN_ROWS, 0, (double)M * D * (4 + es),
           launch_ln_rows(dt, workspace, x_enc, nullptr, ln_g, ln_b, nullptr, M, 1, 0, D, ln_eps,
                          stream));
    LAUNCH(gemm_class(K_GEMM_EMBED, dt, M, D, D), 2.0 * M * (double)D * D,
           es * ((double)M * D + (double)D * D) + 4.0 * (double)M * D + 4.0 * (double)n_tokens * D,
           launch_gemm_embed(dt, workspace, w_de, b_de, M, D, D, x_dec, pe_dec, known, n_enc, n_buf,
                             n_known, n_tokens, stream));
  }
  // algorithmic bytes: the masked rows written, each image position's
  // positional row and the mask token read once (every image reads the same
  // rows), the ranks
  LAUNCH(K_MASK_FILL, 0,
         4.0 * D * ((double)batch * (n_img - n_known) + n_img + 1) + 4.0 * batch * n_img,
         launch_mask_fill(x_dec, mask, pe_dec, rank, batch, n_tokens, n_buf, n_known, D, stream));
  return MARCHE_OK;
}

namespace {

marche_status_t check_head(const marche_head_t *h) {
  if (!h) return fail(MARCHE_ERR_INVALID_ARG, "head is NULL");
  if (raw_enum(h->dtype) != MARCHE_F32 && raw_enum(h->dtype) != MARCHE_BF16)
    return fail(MARCHE_ERR_UNSUPPORTED, "head.dtype=%d is not F32 or BF16", raw_enum(h->dtype));
  if (h->width < 256 || h->width % 256 != 0 || h->width > 4096)
    return fail(MARCHE_ERR_UNSUPPORTED, "head.width=%d (must be a multiple of 256, <= 4096)", h->width);
  if (h->d_cond < 256 || h->d_cond % 256 != 0 || h->d_cond > 4096)
    return fail(MARCHE_ERR_UNSUPPORTED, "head.d_cond=%d (must be a multiple of 256, <= 4096)", h->d_cond);
  if (h->t_freq < 64 || h->t_freq % 64 != 0 || h->t_freq > 4096)
    return fail(MARCHE_ERR_UNSUPPORTED, "head.t_freq=%d (must be a multiple of 64, <= 4096)", h->t_freq);
  if (h->n_blocks < 1 || h->n_blocks > 64)
    return fail(MARCHE_ERR_UNSUPPORTED, "head.n_blocks=%d (supported: 1..64)", h->n_blocks);
  if (h->c_tok < 1 || h->c_tok > 64)
    return fail(MARCHE_ERR_UNSUPPORTED, "head.c_tok=%d (supported: 1..64)", h->c_tok);
  if (!(h->ln_eps > 0.0f)) return fail(MARCHE_ERR_INVALID_ARG, "head.ln_eps must be > 0");
  return MARCHE_OK;
}

// Workspace of the sampler, in carve order.
struct HeadWs {
  size_t z, cond, sinus, h1, temb, sc, mod, h, a, y, t, x, w_in_t, total;
};

HeadWs head_ws(const marche_head_t *hd, int32_t n_rows, int32_t n_steps) {
  const size_t es = elem_size(hd->dtype), M = (size_t)n_rows, T = (size_t)n_steps;
  const size_t W = hd->width, nb = hd->n_blocks;
  HeadWs w{};
  w.z = align256(M * hd->d_cond * es);
  w.cond = align256(M * W * 4);
  w.sinus = align256(T * hd->t_freq * es);
  w.h1 = align256(T * W * es);
  w.temb = align256(T * W * 4);
  w.sc = align256(M * W * es);
  w.mod = align256(M * (3 * nb + 2) * W * es);
  w.h = align256(M * W * 4);
  w.a = align256(M * W * es);
  w.y = align256(M * W * es);
  w.t = align256(M * W * 4);
  w.x = align256(M * hd->c_tok * 4);
  w.w_in_t = align256(W * hd->c_tok * 4);
  w.total = w.z + w.cond + w.sinus + w.h1 + w.temb + w.sc + w.mod + w.h + w.a + w.y + w.t + w.x +
            w.w_in_t;
  return w;
}

}  // namespace

size_t marche_diffusion_workspace_bytes(const marche_head_t *head, int32_t n_rows, int32_t n_steps) {
  if (check_head(head) != MARCHE_OK || n_rows < 0 || n_steps < 1) return 0;
  return head_ws(head, n_rows, n_steps).total;
}

marche_status_t marche_diffusion_sample(const marche_head_t *hd, const marche_head_weights_t *w,
                                        const float *x_dec, int32_t n_tokens, int32_t n_buf,
                                        const float *dec_ln_g, const float *dec_ln_b,
                                        float dec_ln_eps, const float *pe_diff,
                                        const int32_t *rows, const int32_t *out_rows,
                                        int32_t n_rows, const float *noise, int32_t n_steps,
                                        float temperature, float *tok_out, void *workspace,
                                        size_t workspace_bytes, marche_stream_t stream_) {
  marche_status_t st = check_head(hd);
  if (st != MARCHE_OK) return st;
  if (!w) return fail(MARCHE_ERR_INVALID_ARG, "weights are NULL");
  if (n_rows < 0) return fail(MARCHE_ERR_INVALID_ARG, "n_rows=%d < 0", n_rows);
  if (n_steps < 1 || n_steps > 10000)
    return fail(MARCHE_ERR_INVALID_ARG, "n_steps=%d outside [1, 10000]", n_steps);
  if (n_tokens < 1 || n_buf < 0 || n_buf >= n_tokens)
    return fail(MARCHE_ERR_INVALID_ARG, "n_tokens=%d n_buf=%d inconsistent", n_tokens, n_buf);
  if (!(dec_ln_eps > 0.0f)) return fail(MARCHE_ERR_INVALID_ARG, "dec_ln_eps must be > 0");
  if (!(temperature >= 0.0f) || temperature > 1e30f)
    return fail(MARCHE_ERR_INVALID_ARG, "temperature must be finite and >= 0");
  const int W = hd->width, nb = hd->n_blocks, C = hd->c_tok, D = hd->d_cond, F = hd->t_freq;
  const int ML = (3 * nb + 2) * W;
  // GEMM epilogues use 32-bit element offsets
  if ((int64_t)n_rows * ML >= (1LL << 31) || (int64_t)n_rows * D >= (1LL << 31) ||
      (int64_t)n_steps * std::max(W, F) >= (1LL << 31))
    return fail(MARCHE_ERR_UNSUPPORTED, "sampler buffers reach 2^31 elements");
  if (n_rows == 0) return MARCHE_OK;
  const void *wp[] = {w->w_t1, w->b_t1, w->w_t2, w->b_t2, w->w_c, w->b_c, w->w_in, w->b_in,
                      w->w_ada, w->b_ada, w->w_1, w->b_1, w->w_2, w->b_2, w->w_out, w->b_out};
  for (const void *q : wp)
    if (!q) return fail(MARCHE_ERR_INVALID_ARG, "a head weight is NULL");
  if (!x_dec || !dec_ln_g || !dec_ln_b || !pe_diff || !rows || !out_rows || !noise || !tok_out)
    return fail(MARCHE_ERR_INVALID_ARG, "NULL input to marche_diffusion_sample");
  const HeadWs L = head_ws(hd, n_rows, n_steps);
  if (!workspace || workspace_bytes < L.total)
    return fail(MARCHE_ERR_WORKSPACE, "workspace %s: %zu bytes < %zu needed",
                workspace ? "too small" : "is NULL", workspace_bytes, L.total);
  if (reinterpret_cast<uintptr_t>(workspace) & 255)
    return fail(MARCHE_ERR_INVALID_ARG, "workspace must be 256-byte aligned");

  hipStream_t stream = static_cast<hipStream_t>(stream_);
  const DType dt = hd->dtype == MARCHE_BF16 ? DType::BF16 : DType::F32;
  const size_t es = elem_size(hd->dtype);
  const int M = n_rows, T = n_steps;
  char *p = static_cast<char *>(workspace);
  auto take = [&](size_t n) { char *q = p; p += n; return q; };
  void *z = take(L.z);
  float *cond = reinterpret_cast<float *>(take(L.cond));
  void *sinus = take(L.sinus);
  void *h1 = take(L.h1);
  float *temb = reinterpret_cast<float *>(take(L.temb));
  void *sc = take(L.sc);
  void *mod = take(L.mod);
  float *hbuf = reinterpret_cast<float *>(take(L.h));
  void *abuf = take(L.a);
  void *ybuf = take(L.y);
  float *tbuf = reinterpret_cast<float *>(take(L.t));
  float *xs = reinterpret_cast<float *>(take(L.x));
  float *w_in_t = reinterpret_cast<float *>(take(L.w_in_t));
  auto fp = [](const void *q) { return static_cast<const float *>(q); };

  LAUNCH(K_TRANSPOSE, 0, 8.0 * W * C,
         launch_transpose_f32(w_in_t, fp(w->w_in), W, C, stream));
  // condition rows and the time-embedding table (all timesteps)
  LAUNCH(K_LN_ROWS, 0, (double)M * D * (4 + es) + 4.0 * M * D,
         launch_ln_rows(dt, z, x_dec, rows, dec_ln_g, dec_ln_b, pe_diff, M, n_tokens, n_buf, D,
                        dec_ln_eps, stream));
  LAUNCH(gemm_class(K_GEMM_HEAD, dt, M, W, D), 2.0 * M * (double)W * D,
         es * ((double)M * D + (double)W * D) + 4.0 * M * W,
         launch_gemm_plain(dt, z, w->w_c, fp(w->b_c), M, W, D, cond, DType::F32, false, stream));
  LAUNCH(K_TIME_SINUS, 0, es * (double)T * F, launch_time_sinus(dt, sinus, T, F, stream));
  LAUNCH(gemm_class(K_GEMM_HEAD_SILU, dt, T, W, F), 2.0 * T * (double)W * F,
         es * ((double)T * F + (double)W * F + (double)T * W),
         launch_gemm_plain(dt, sinus, w->w_t1, fp(w->b_t1), T, W, F, h1, dt, true, stream));
  LAUNCH(gemm_class(K_GEMM_HEAD, dt, T, W, W), 2.0 * T * (double)W * W,
         es * ((double)T * W + (double)W * W) + 4.0 * T * W,
         launch_gemm_plain(dt, h1, w->w_t2, fp(w->b_t2), T, W, W, temb, DType::F32, false, stream));

  // cosine schedule (double precision on the host)
  std::vector<double> betas(T), abar(T);
  {
    auto g = [](double u) {
      const double c = std::cos((u + 0.008) / 1.008 * 1.5707963267948966);
      return c * c;
    };
    double prod = 1.0;
    for (int i = 0; i < T; ++i) {
      betas[i] = std::min(1.0 - g((double)(i + 1) / T) / g((double)i / T), 0.999);
      prod *= 1.0 - betas[i];
      abar[i] = prod;
    }
  }
  const float *x_init = noise + (size_t)T * M * C;
  for (int i = T - 1; i >= 0; --i) {
    const float *xc = i == T - 1 ? x_init : xs;
    LAUNCH(K_HEAD_SILU_COND, 0, 4.0 * M * W + es * (double)M * W,
           launch_silu_cond(dt, sc, cond, temb + (size_t)i * W, M, W, stream));
    LAUNCH(gemm_class(K_GEMM_HEAD, dt, M, ML, W), 2.0 * M * (double)ML * W,
           es * ((double)M * W + (double)ML * W + (double)M * ML),
           launch_gemm_plain(dt, sc, w->w_ada, fp(w->b_ada), M, ML, W, mod, dt, false, stream));
    LAUNCH(K_HEAD_IN_MOD, 2.0 * M * (double)W * C,
           4.0 * M * C + 4.0 * M * W + es * 3.0 * M * W,
           launch_head_in_mod(dt, abuf, hbuf, xc, w_in_t, fp(w->b_in), mod, ML, M, W, C,
                              hd->ln_eps, stream));
    for (int k = 0; k < nb; ++k) {
      const char *w1 = static_cast<const char *>(w->w_1) + (size_t)k * W * W * es;
      const char *w2 = static_cast<const char *>(w->w_2) + (size_t)k * W * W * es;
      LAUNCH(gemm_class(K_GEMM_HEAD_SILU, dt, M, W, W), 2.0 * M * (double)W * W,
             es * (2.0 * M * W + (double)W * W),
             launch_gemm_plain(dt, abuf, w1, fp(w->b_1) + (size_t)k * W, M, W, W, ybuf, dt, true,
                               stream));
      LAUNCH(gemm_class(K_GEMM_HEAD, dt, M, W, W), 2.0 * M * (double)W * W,
             es * ((double)M * W + (double)W * W) + 4.0 * M * W,
             launch_gemm_plain(dt, ybuf, w2, fp(w->b_2) + (size_t)k * W, M, W, W, tbuf,
                               DType::F32, false, stream));
      // the next modulated norm: block k + 1's, or the final layer's
      const int nxt = 3 * (k + 1) * W;
      LAUNCH(K_HEAD_GATE_MOD, 0, 4.0 * 3.0 * M * W + es * 4.0 * M * W,
             launch_head_gate_mod(dt, abuf, hbuf, tbuf, mod, ML, 3 * k * W + 2 * W, nxt, nxt + W,
                                  M, W, hd->ln_eps, stream));
    }
    const double ab = abar[i], abp = i > 0 ? abar[i - 1] : 1.0, b = betas[i];
    HeadStep hs;
    hs.sra = (float)(1.0 / std::sqrt(ab));
    hs.srm1 = (float)std::sqrt(1.0 / ab - 1.0);
    hs.c1 = (float)(b * std::sqrt(abp) / (1.0 - ab));
    hs.c2 = (float)((1.0 - abp) * std::sqrt(1.0 - b) / (1.0 - ab));
    hs.sigma = i > 0 ? (float)(temperature * std::sqrt(b * (1.0 - abp) / (1.0 - ab))) : 0.0f;
    LAUNCH(K_HEAD_OUT_STEP, 2.0 * M * (double)W * C,
           es * (double)M * W + 4.0 * ((double)C * W + 3.0 * M * C),
           launch_head_out_step(dt, xs, i == 0 ? tok_out : nullptr, abuf, fp(w->w_out),
                                fp(w->b_out), xc, noise + (size_t)i * M * C, out_rows, M, W, C,
                                hs, stream));
  }
  return MARCHE_OK;
}

marche_status_t marche_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_prof = on != 0;
  return MARCHE_OK;
}

int32_t marche_profile_collect(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (Pending &p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.e1) == hipSuccess && hipEventElapsedTime(&ms, p.e0, p.e1) == hipSuccess) {
      Totals &t = g_tot[p.cls];
      t.launches += 1;
      t.ms += ms;
      t.flops += p.flops;
      t.bytes += p.bytes;
    }
    g_pool.push_back(p.e0);
    g_pool.push_back(p.e1);
  }
  g_pending.clear();
  return K_NTIMED;
}

marche_status_t marche_profile_entry(int32_t i, const char **name, int64_t *launches,
                                     double *total_ms, double *flops, double *bytes) {
  if (i < 0 || i >= K_NTIMED) return fail(MARCHE_ERR_INVALID_ARG, "profile entry %d out of range", i);
  std::lock_guard<std::mutex> lk(g_mu);
  const Totals &t = g_tot[i];
  if (name) *name = class_name(i);
  if (launches) *launches = t.launches;
  if (total_ms) *total_ms = t.ms;
  if (flops) *flops = t.flops;
  if (bytes) *bytes = t.bytes;
  return MARCHE_OK;
}

void marche_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (Pending &p : g_pending) {
    g_pool.push_back(p.e0);
    g_pool.push_back(p.e1);
  }
  g_pending.clear();
  for (Totals &t : g_tot) t = Totals();
}

}  // extern "C"
