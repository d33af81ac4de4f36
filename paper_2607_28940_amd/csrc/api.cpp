// C ABI of the TransX serving path: model repack, paged KV cache bookkeeping,
// work planning and the launch sequence of kv_cache_build, kv_cache_append and
// score_candidates. Host code only; every computation step runs in the HIP
// kernels of gemm.hip, attention.hip and rowops.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#pragma GCC visibility push(default)
#include "transx.h"
#pragma GCC visibility pop

#include "tx_internal.h"
#include "xplan.h"

using namespace tx;

// ------------------------------------------------------------------ errors
namespace {
thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define TX_HIP(expr)                                                                        \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return fail(TX_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define TX_CHECK(code)           \
  do {                           \
    int c_ = (code);             \
    if (c_ != TX_OK) return c_;  \
  } while (0)

size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// Pinned staging per ring slot reserved when a cache is created: the largest
// per-pass metadata score_candidates_static uploads (its passes are planned
// to fit).
constexpr size_t kStagingReserve = 512 << 10;

// Lays sub-buffers out in one device region (256-byte aligned); with a null
// base it only measures.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  template <class P>
  P take(size_t bytes) {
    const size_t o = align_up(off);
    off = o + bytes;
    return base ? (P)(base + o) : (P) nullptr;
  }
};
}  // namespace

// ------------------------------------------------------------------ model
namespace {
struct Mat {
  void* w = nullptr;  // [N][K] transposed weight, model dtype
  float* b = nullptr; // [N] fp32 bias
  int N = 0, K = 0;
};
struct EncLayer {
  Mat qkv, o, f1, f2;
  float *ln1g, *ln1b, *ln2g, *ln2b, *rel;
};
// A consumer GEMM with the preceding LayerNorm folded in (bf16 models, see
// EPI_LN in tx_internal.h): gain-scaled weight [N][K] in fp16, its column sums
// and the bias with the LayerNorm offset folded in.
struct Fold {
  void* w = nullptr;
  float* cs = nullptr;
  float* b = nullptr;
};
struct DecLayer {
  Mat qkv, o, xq, xo, f1, f2;
  float *ln1g, *ln1b, *ln2g, *ln2b, *ln3g, *ln3b;
  // cross-Q with LN1, FFN up with LN2, and (layers after the first) QKV with
  // the previous layer's LN3 folded in
  Fold xqf, f1f, qkvf;
};
enum { E_WQ, E_BQ, E_WK, E_BK, E_WV, E_BV, E_WO, E_BO, E_LN1G, E_LN1B, E_W1, E_B1, E_W2, E_B2, E_LN2G, E_LN2B,
       E_REL, E_N };
enum { D_SWQ, D_SBQ, D_SWK, D_SBK, D_SWV, D_SBV, D_SWO, D_SBO, D_LN1G, D_LN1B, D_XWQ, D_XBQ, D_XWK, D_XBK, D_XWV,
       D_XBV, D_XWO, D_XBO, D_LN2G, D_LN2B, D_W1, D_B1, D_W2, D_B2, D_LN3G, D_LN3B, D_N };
}  // namespace

struct tx_model {
  tx_config cfg;
  uint64_t id;
  bool bf;
  int d, H, dh, F, n_enc, n_dec, R;
  size_t esz;
  std::vector<EncLayer> enc;
  std::vector<DecLayer> dec;
  Mat xkv;  // cross-attention K and V of every decoder layer: [n_dec * 2d][d]
  float* ws;
  float* bs;
  float* wpool = nullptr;  // attention-pooling vector of the global token [d]
  int l_local = 0;         // > 0: local-global sparse cross-attention
  bool gpool = false;      // the sparse key set includes the pooled global token
  int n_act = 0;           // 0: scalar logit head (ws [d], bs [1]); k: ws [k][d], bs [k]
  bool weights_set = false;
  bool ln_fold = false;    // bf16: the folded weights exist and are finite in fp16
  int* fold_flag = nullptr;  // device word: a folded weight overflowed fp16
};

static int check_config(const tx_config* c) {
  if (!c) return fail(TX_E_INVALID, "config is null");
  if (c->dtype != TX_F32 && c->dtype != TX_BF16) return fail(TX_E_INVALID, "dtype %d unknown", c->dtype);
  if (c->d_model <= 0 || c->n_heads <= 0 || c->d_model % c->n_heads)
    return fail(TX_E_INVALID, "d_model %d must be a positive multiple of n_heads %d", c->d_model, c->n_heads);
  const int dh = c->d_model / c->n_heads;
  if (dh != 32 && dh != 64 && dh != 128) return fail(TX_E_UNSUPPORTED, "d_head %d not in {32, 64, 128}", dh);
  if (c->d_ffn <= 0) return fail(TX_E_INVALID, "d_ffn %d", c->d_ffn);
  if (c->n_enc_layers < 1 || c->n_dec_layers < 1 || c->n_enc_layers > 64 || c->n_dec_layers > 64)
    return fail(TX_E_INVALID, "layer counts enc %d dec %d", c->n_enc_layers, c->n_dec_layers);
  if (c->rel_pos_buckets < 0) return fail(TX_E_INVALID, "rel_pos_buckets %d", c->rel_pos_buckets);
  if (!(c->ln_eps > 0.f)) return fail(TX_E_INVALID, "ln_eps must be positive");
  if (c->l_local < 0) return fail(TX_E_INVALID, "l_local %d", c->l_local);
  if (c->l_local > kMaxLocal) return fail(TX_E_UNSUPPORTED, "l_local %d above %d", c->l_local, kMaxLocal);
  if (c->global_pool != 0 && c->global_pool != 1) return fail(TX_E_INVALID, "global_pool %d", c->global_pool);
  if (c->global_pool && c->l_local == 0)
    return fail(TX_E_INVALID, "the pooled global token belongs to the sparse cross-attention (l_local > 0)");
  if (c->n_actions < 0 || c->n_actions == 1) return fail(TX_E_INVALID, "n_actions %d (0 or >= 2)", c->n_actions);
  if (c->n_actions > kMaxActions) return fail(TX_E_UNSUPPORTED, "n_actions %d above %d", c->n_actions, kMaxActions);
  return TX_OK;
}

static void layout_model(const tx_config& c, Carver& cv, tx_model& m) {
  const int d = c.d_model, F = c.d_ffn, H = c.n_heads, R = c.rel_pos_buckets;
  const size_t es = c.dtype == TX_BF16 ? 2 : 4;
  auto mat = [&](int N, int K) {
    Mat x;
    x.N = N;
    x.K = K;
    x.w = cv.take<void*>((size_t)N * K * es);
    x.b = cv.take<float*>((size_t)N * 4);
    return x;
  };
  auto vec = [&](size_t n) { return cv.take<float*>(std::max<size_t>(n, 1) * 4); };
  m.enc.resize(c.n_enc_layers);
  for (auto& L : m.enc) {
    L.qkv = mat(3 * d, d);
    L.o = mat(d, d);
    L.f1 = mat(F, d);
    L.f2 = mat(d, F);
    L.ln1g = vec(d), L.ln1b = vec(d), L.ln2g = vec(d), L.ln2b = vec(d);
    L.rel = vec((size_t)H * R);
  }
  auto fold = [&](int N, int K) {
    Fold x;
    x.w = cv.take<void*>((size_t)N * K * 2);
    x.cs = vec(N);
    x.b = vec(N);
    return x;
  };
  m.dec.resize(c.n_dec_layers);
  for (int l = 0; l < c.n_dec_layers; ++l) {
    DecLayer& L = m.dec[l];
    L.qkv = mat(3 * d, d);
    L.o = mat(d, d);
    L.xq = mat(d, d);
    L.xo = mat(d, d);
    L.f1 = mat(F, d);
    L.f2 = mat(d, F);
    L.ln1g = vec(d), L.ln1b = vec(d), L.ln2g = vec(d), L.ln2b = vec(d), L.ln3g = vec(d), L.ln3b = vec(d);
    if (c.dtype == TX_BF16) {
      L.xqf = fold(d, d);
      L.f1f = fold(F, d);
      if (l > 0) L.qkvf = fold(3 * d, d);
    }
  }
  if (c.dtype == TX_BF16) m.fold_flag = cv.take<int*>(sizeof(int));
  m.xkv = mat(2 * d * c.n_dec_layers, d);
  const int k = std::max(1, c.n_actions);
  m.ws = vec((size_t)d * k);
  m.bs = vec(k);
  if (c.global_pool) m.wpool = vec(d);
}

extern "C" {

const char* tx_last_error(void) { return g_err.c_str(); }

int32_t tx_num_weights(const tx_config* cfg) {
  if (!cfg) return -1;
  return E_N * cfg->n_enc_layers + D_N * cfg->n_dec_layers + 2 + (cfg->global_pool ? 1 : 0);
}

size_t tx_model_repack_bytes(const tx_config* cfg) {
  if (check_config(cfg) != TX_OK) return 0;
  tx_model m;
  Carver cv(nullptr);
  layout_model(*cfg, cv, m);
  return align_up(cv.off);
}

int tx_model_create(const tx_config* cfg, void* dev_repack, size_t repack_bytes, uint64_t model_id, tx_model** out) {
  if (!out) return fail(TX_E_INVALID, "out is null");
  *out = nullptr;
  TX_CHECK(check_config(cfg));
  const size_t need = tx_model_repack_bytes(cfg);
  if (!dev_repack || ((uintptr_t)dev_repack & 255)) return fail(TX_E_INVALID, "repack buffer null or not 256-byte aligned");
  if (repack_bytes < need) return fail(TX_E_NOMEM, "repack buffer %zu bytes < %zu", repack_bytes, need);
  tx_model* m = new tx_model();
  m->cfg = *cfg;
  m->id = model_id;
  m->bf = cfg->dtype == TX_BF16;
  m->d = cfg->d_model;
  m->H = cfg->n_heads;
  m->dh = cfg->d_model / cfg->n_heads;
  m->F = cfg->d_ffn;
  m->n_enc = cfg->n_enc_layers;
  m->n_dec = cfg->n_dec_layers;
  m->R = cfg->rel_pos_buckets;
  m->esz = m->bf ? 2 : 4;
  m->l_local = cfg->l_local;
  m->gpool = cfg->global_pool != 0;
  m->n_act = cfg->n_actions;
  Carver cv(dev_repack);
  layout_model(*cfg, cv, *m);
  *out = m;
  return TX_OK;
}

int tx_model_set_weights(tx_model* m, const void* const* W, int32_t n_weights, hipStream_t stream) {
  if (!m) return fail(TX_E_INVALID, "model is null");
  const tx_config* cfg = &m->cfg;
  if (n_weights != tx_num_weights(cfg))
    return fail(TX_E_INVALID, "expected %d weight tensors, got %d", tx_num_weights(cfg), n_weights);
  if (!W) return fail(TX_E_INVALID, "weights array is null");
  for (int i = 0; i < n_weights; ++i) {
    const bool empty_rel = (i < E_N * cfg->n_enc_layers) && (i % E_N == E_REL) && cfg->rel_pos_buckets == 0;
    if (!W[i] && !empty_rel) return fail(TX_E_INVALID, "weight tensor %d is null", i);
    if (W[i] && ((uintptr_t)W[i] % m->esz)) return fail(TX_E_INVALID, "weight tensor %d misaligned", i);
  }
  const int d = m->d, F = m->F;
  const bool bf = m->bf;
  const size_t es = m->esz;
  auto wp = [&](int i) { return W[i]; };
  auto tr = [&](int i, void* dst, int K, int N, int dst_ld) { return launch_transpose(bf, wp(i), dst, K, N, dst_ld, stream); };
  auto bias = [&](int i, float* dst, int64_t n) { return launch_to_f32(bf, wp(i), dst, n, stream); };
  auto at = [&](void* base, size_t elems) { return (void*)((char*)base + elems * es); };
  hipError_t e = hipSuccess;
  auto run = [&](hipError_t x) { if (e == hipSuccess) e = x; };
  for (int l = 0; l < m->n_enc; ++l) {
    const int b = l * E_N;
    EncLayer& L = m->enc[l];
    run(tr(b + E_WQ, L.qkv.w, d, d, d));
    run(tr(b + E_WK, at(L.qkv.w, (size_t)d * d), d, d, d));
    run(tr(b + E_WV, at(L.qkv.w, (size_t)2 * d * d), d, d, d));
    run(bias(b + E_BQ, L.qkv.b, d));
    run(bias(b + E_BK, L.qkv.b + d, d));
    run(bias(b + E_BV, L.qkv.b + 2 * d, d));
    run(tr(b + E_WO, L.o.w, d, d, d));
    run(bias(b + E_BO, L.o.b, d));
    run(tr(b + E_W1, L.f1.w, d, F, d));
    run(bias(b + E_B1, L.f1.b, F));
    run(tr(b + E_W2, L.f2.w, F, d, F));
    run(bias(b + E_B2, L.f2.b, d));
    run(bias(b + E_LN1G, L.ln1g, d));
    run(bias(b + E_LN1B, L.ln1b, d));
    run(bias(b + E_LN2G, L.ln2g, d));
    run(bias(b + E_LN2B, L.ln2b, d));
    if (m->R > 0) run(bias(b + E_REL, L.rel, (int64_t)m->H * m->R));
  }
  for (int l = 0; l < m->n_dec; ++l) {
    const int b = E_N * m->n_enc + l * D_N;
    DecLayer& L = m->dec[l];
    run(tr(b + D_SWQ, L.qkv.w, d, d, d));
    run(tr(b + D_SWK, at(L.qkv.w, (size_t)d * d), d, d, d));
    run(tr(b + D_SWV, at(L.qkv.w, (size_t)2 * d * d), d, d, d));
    run(bias(b + D_SBQ, L.qkv.b, d));
    run(bias(b + D_SBK, L.qkv.b + d, d));
    run(bias(b + D_SBV, L.qkv.b + 2 * d, d));
    run(tr(b + D_SWO, L.o.w, d, d, d));
    run(bias(b + D_SBO, L.o.b, d));
    run(tr(b + D_XWQ, L.xq.w, d, d, d));
    run(bias(b + D_XBQ, L.xq.b, d));
    run(tr(b + D_XWK, at(m->xkv.w, (size_t)(2 * l) * d * d), d, d, d));
    run(tr(b + D_XWV, at(m->xkv.w, (size_t)(2 * l + 1) * d * d), d, d, d));
    run(bias(b + D_XBK, m->xkv.b + (size_t)(2 * l) * d, d));
    run(bias(b + D_XBV, m->xkv.b + (size_t)(2 * l + 1) * d, d));
    run(tr(b + D_XWO, L.xo.w, d, d, d));
    run(bias(b + D_XBO, L.xo.b, d));
    run(tr(b + D_W1, L.f1.w, d, F, d));
    run(bias(b + D_B1, L.f1.b, F));
    run(tr(b + D_W2, L.f2.w, F, d, F));
    run(bias(b + D_B2, L.f2.b, d));
    run(bias(b + D_LN1G, L.ln1g, d));
    run(bias(b + D_LN1B, L.ln1b, d));
    run(bias(b + D_LN2G, L.ln2g, d));
    run(bias(b + D_LN2B, L.ln2b, d));
    run(bias(b + D_LN3G, L.ln3g, d));
    run(bias(b + D_LN3B, L.ln3b, d));
  }
  const int hb = E_N * m->n_enc + D_N * m->n_dec;
  const int k = std::max(1, m->n_act);
  if (m->n_act) run(launch_transpose_to_f32(bf, wp(hb), m->ws, d, k, stream));  // W_dec [d][k] -> [k][d]
  else run(bias(hb, m->ws, d));
  run(bias(hb + 1, m->bs, k));
  if (m->gpool) run(bias(hb + 2, m->wpool, d));
  // the LayerNorm folds of the bf16 score pass; they stay unused when a
  // gain-scaled weight does not fit fp16 (read back once, here)
  m->ln_fold = false;
  if (bf) {
    run(launch_zero_int(m->fold_flag, stream));
    for (int l = 0; l < m->n_dec; ++l) {
      DecLayer& L = m->dec[l];
      run(launch_fold_ln_weight(L.xq.w, d, d, L.ln1g, L.ln1b, L.xq.b, L.xqf.w, L.xqf.cs, L.xqf.b, m->fold_flag, stream));
      run(launch_fold_ln_weight(L.f1.w, F, d, L.ln2g, L.ln2b, L.f1.b, L.f1f.w, L.f1f.cs, L.f1f.b, m->fold_flag, stream));
      if (l > 0)
        run(launch_fold_ln_weight(L.qkv.w, 3 * d, d, m->dec[l - 1].ln3g, m->dec[l - 1].ln3b, L.qkv.b, L.qkvf.w,
                                  L.qkvf.cs, L.qkvf.b, m->fold_flag, stream));
    }
  }
  if (e != hipSuccess) return fail(TX_E_HIP, "weight repack launch failed: %s", hipGetErrorString(e));
  if (bf) {
    int flag = 1;
    e = read_int(m->fold_flag, &flag, stream);
    if (e != hipSuccess) return fail(TX_E_HIP, "weight fold check failed: %s", hipGetErrorString(e));
    m->ln_fold = flag == 0;
  }
  m->weights_set = true;
  return TX_OK;
}

void tx_model_destroy(tx_model* m) { delete m; }

}  // extern "C"

// ------------------------------------------------------------------ cache
namespace {
// Pinned host staging for small metadata uploads: a ring of buffers, each
// reused only after the copy that last read it has completed.
struct Stager {
  struct Slot {
    char* host = nullptr;
    size_t cap = 0;
    hipEvent_t ev = nullptr;
    bool pending = false;
  };
  Slot slot[4];
  int next = 0;
  ~Stager() {
    for (auto& s : slot) {
      if (s.pending) (void)hipEventSynchronize(s.ev);
      if (s.ev) (void)hipEventDestroy(s.ev);
      if (s.host) (void)hipHostFree(s.host);
    }
  }
  // Gives every slot an event and at least `cap` bytes of pinned memory.
  hipError_t reserve(size_t cap) {
    for (int i = 0; i < 4; ++i) {
      Slot* s = nullptr;
      hipError_t e = acquire(cap, &s, true);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  // The next slot of the ring, grown to n bytes if may_grow (a slot too small
  // otherwise is hipErrorOutOfMemory: nothing is allocated).
  hipError_t acquire(size_t n, Slot** out, bool may_grow) {
    Slot& s = slot[next];
    if (!may_grow && (s.cap < n || !s.ev)) return hipErrorOutOfMemory;
    next = (next + 1) & 3;
    if (s.pending) {
      hipError_t e = hipEventSynchronize(s.ev);
      if (e != hipSuccess) return e;
      s.pending = false;
    }
    if (!s.ev) {
      hipError_t e = hipEventCreateWithFlags(&s.ev, hipEventDisableTiming);
      if (e != hipSuccess) return e;
    }
    if (s.cap < n) {
      if (s.host) (void)hipHostFree(s.host);
      s.host = nullptr;
      s.cap = 0;
      const size_t c = std::max<size_t>(align_up(n, 65536), 65536);
      hipError_t e = hipHostMalloc((void**)&s.host, c, hipHostMallocDefault);
      if (e != hipSuccess) return e;
      s.cap = c;
    }
    *out = &s;
    return hipSuccess;
  }
  hipError_t upload(void* dst, const void* src, size_t n, hipStream_t st, bool may_grow = true) {
    if (n == 0) return hipSuccess;
    Slot* s = nullptr;
    hipError_t e = acquire(n, &s, may_grow);
    if (e != hipSuccess) return e;
    memcpy(s->host, src, n);
    e = hipMemcpyAsync(dst, s->host, n, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return e;
    e = hipEventRecord(s->ev, st);
    if (e != hipSuccess) return e;
    s->pending = true;
    return hipSuccess;
  }
};
}  // namespace

struct tx_kv_cache {
  const tx_model* m;
  char* pool;
  size_t pool_bytes;
  int64_t n_pages;
  int32_t max_req;
  int64_t max_tokens;
  int32_t max_pages;  // pages per request
  size_t page_bytes;
  PageGeom geom;
  int32_t* d_table;  // device [max_req][max_pages]
  // global token of the sparse cross-attention, per page-table row: pooling
  // state (max, sum) and weighted row sum (fp32), and its cross K/V rows
  // [n_dec * 2d] in the model dtype (layer l: K at 2l*d, V at (2l+1)*d)
  float* d_pool_ml = nullptr;
  float* d_pool_acc = nullptr;
  char* d_gkv = nullptr;
  std::vector<int32_t> h_table;
  std::vector<std::vector<int32_t>> pages;
  std::vector<int64_t> len;  // -1: no cache
  std::vector<int32_t> free_list;
  mutable Stager st;  // metadata uploads also happen in const (score) calls
  bool staging_reserved = false;  // the ring holds kStagingReserve bytes per slot
};

extern "C" {

size_t tx_kv_page_bytes(const tx_config* c) {
  if (check_config(c) != TX_OK) return 0;
  const size_t es = c->dtype == TX_BF16 ? 2 : 4;
  return (size_t)(c->n_enc_layers + c->n_dec_layers) * 2 * kPage * c->d_model * es;
}

// Bytes of the per-request global-token records that follow the page table.
static size_t global_token_bytes(const tx_config* c, int64_t max_requests) {
  if (!c->global_pool) return 0;
  const size_t es = c->dtype == TX_BF16 ? 2 : 4, d = c->d_model;
  return align_up((size_t)max_requests * 2 * 4) + align_up((size_t)max_requests * d * 4) +
         align_up((size_t)max_requests * 2 * c->n_dec_layers * d * es);
}

size_t tx_kv_pool_bytes(const tx_config* c, int64_t n_pages, int32_t max_requests, int64_t max_tokens) {
  if (check_config(c) != TX_OK || n_pages < 0 || max_requests < 0 || max_tokens < 0) return 0;
  const int64_t mp = (max_tokens + kPage - 1) / kPage;
  return align_up((size_t)n_pages * tx_kv_page_bytes(c)) + align_up((size_t)max_requests * mp * 4) +
         global_token_bytes(c, max_requests);
}

int tx_kv_cache_create(const tx_model* m, void* dev_pool, size_t pool_bytes, int64_t n_pages, int32_t max_requests,
                       int64_t max_tokens, tx_kv_cache** out) {
  if (!out) return fail(TX_E_INVALID, "out is null");
  *out = nullptr;
  if (!m) return fail(TX_E_INVALID, "model is null");
  if (n_pages < 1 || n_pages > INT32_MAX) return fail(TX_E_INVALID, "n_pages %lld", (long long)n_pages);
  if (max_requests < 1) return fail(TX_E_INVALID, "max_requests %d", max_requests);
  if (max_tokens < 1 || max_tokens > (int64_t)1 << 30) return fail(TX_E_INVALID, "max_tokens %lld", (long long)max_tokens);
  if (!dev_pool || ((uintptr_t)dev_pool & 255)) return fail(TX_E_INVALID, "pool null or not 256-byte aligned");
  const size_t need = tx_kv_pool_bytes(&m->cfg, n_pages, max_requests, max_tokens);
  if (pool_bytes < need) return fail(TX_E_NOMEM, "pool %zu bytes < %zu needed", pool_bytes, need);
  tx_kv_cache* c = new tx_kv_cache();
  c->m = m;
  c->pool = (char*)dev_pool;
  c->pool_bytes = pool_bytes;
  c->n_pages = n_pages;
  c->max_req = max_requests;
  c->max_tokens = max_tokens;
  c->max_pages = (int32_t)((max_tokens + kPage - 1) / kPage);
  c->page_bytes = tx_kv_page_bytes(&m->cfg);
  c->geom.H = m->H;
  c->geom.dh = m->dh;
  c->geom.n_slots = m->n_enc + m->n_dec;
  c->geom.page_elems = (int64_t)(c->page_bytes / m->esz);
  c->d_table = (int32_t*)(c->pool + align_up((size_t)n_pages * c->page_bytes));
  if (m->gpool) {
    char* p = (char*)c->d_table + align_up((size_t)max_requests * c->max_pages * 4);
    c->d_pool_ml = (float*)p;
    p += align_up((size_t)max_requests * 2 * 4);
    c->d_pool_acc = (float*)p;
    p += align_up((size_t)max_requests * m->d * 4);
    c->d_gkv = p;
  }
  c->h_table.assign((size_t)max_requests * c->max_pages, 0);
  c->pages.resize(max_requests);
  c->len.assign(max_requests, -1);
  c->free_list.resize(n_pages);
  for (int64_t i = 0; i < n_pages; ++i) c->free_list[i] = (int32_t)(n_pages - 1 - i);  // pop_back gives page 0 first
  // pinned staging for the metadata of score_candidates_static, which may not
  // allocate; without a usable device that call reports TX_E_NOMEM instead
  c->staging_reserved = c->st.reserve(kStagingReserve) == hipSuccess;
  if (!c->staging_reserved) (void)hipGetLastError();
  *out = c;
  return TX_OK;
}

void tx_kv_cache_destroy(tx_kv_cache* c) { delete c; }

int tx_kv_cache_release(tx_kv_cache* c, int32_t n_req, const int32_t* ids) {
  if (!c) return fail(TX_E_INVALID, "cache is null");
  if (n_req < 0 || (n_req > 0 && !ids)) return fail(TX_E_INVALID, "bad id list");
  for (int i = 0; i < n_req; ++i)
    if (ids[i] < 0 || ids[i] >= c->max_req) return fail(TX_E_INVALID, "request id %d out of range", ids[i]);
  for (int i = 0; i < n_req; ++i) {
    auto& pg = c->pages[ids[i]];
    for (int32_t p : pg) c->free_list.push_back(p);
    pg.clear();
    c->len[ids[i]] = -1;
  }
  return TX_OK;
}

int tx_kv_cache_length(const tx_kv_cache* c, int32_t id, int64_t* len_out) {
  if (!c || !len_out) return fail(TX_E_INVALID, "null argument");
  if (id < 0 || id >= c->max_req) return fail(TX_E_INVALID, "request id %d out of range", id);
  *len_out = c->len[id];
  return TX_OK;
}

int64_t tx_kv_cache_free_pages(const tx_kv_cache* c) { return c ? (int64_t)c->free_list.size() : -1; }

uint64_t tx_kv_cache_model_id(const tx_kv_cache* c) { return c ? c->m->id : 0; }

int tx_kv_cache_export(const tx_kv_cache* c, int32_t id, int32_t part, int32_t layer, void* out, hipStream_t stream) {
  if (!c || !out) return fail(TX_E_INVALID, "null argument");
  if (id < 0 || id >= c->max_req) return fail(TX_E_INVALID, "request id %d out of range", id);
  if (c->len[id] < 0) return fail(TX_E_NOCACHE, "request %d has no cache", id);
  if (part < 0 || part > 5) return fail(TX_E_INVALID, "part %d", part);
  if (part >= 4) {  // the global token's cross-attention key (4) or value (5)
    if (!c->m->gpool) return fail(TX_E_INVALID, "model has no pooled global token");
    if (layer < 0 || layer >= c->m->n_dec) return fail(TX_E_INVALID, "layer %d", layer);
    const size_t es = c->m->esz, d = c->m->d;
    const char* src = c->d_gkv + ((size_t)id * 2 * c->m->n_dec * d + (size_t)(2 * layer + (part - 4)) * d) * es;
    TX_HIP(hipMemcpyAsync(out, src, d * es, hipMemcpyDeviceToDevice, stream));
    return TX_OK;
  }
  if (c->len[id] == 0) return TX_OK;
  const int nl = part < 2 ? c->m->n_enc : c->m->n_dec;
  if (layer < 0 || layer >= nl) return fail(TX_E_INVALID, "layer %d", layer);
  const int slot = part < 2 ? layer : c->m->n_enc + layer;
  TX_HIP(launch_export_kv(c->m->bf, c->pool, c->d_table + (size_t)id * c->max_pages, c->geom, slot, part & 1,
                          c->len[id], out, stream));
  return TX_OK;
}

}  // extern "C"


// ------------------------------------------------------------------ kernel timing
namespace {
enum KClass {
  K_GEMM_QKV, K_GEMM_O, K_GEMM_XQ, K_GEMM_XO, K_GEMM_FFN1, K_GEMM_FFN2, K_SELF_ATTN, K_CROSS_ATTN, K_LAYERNORM,
  K_LN_SCORE, K_COPY, K_ENC_GEMM, K_ENC_ATTN, K_ENC_LAYERNORM, K_SCATTER, K_XKV_GEMM, K_POOL, K_COUNT
};
const char* const kClassNames[K_COUNT] = {
    "score.gemm_qkv", "score.gemm_self_out", "score.gemm_cross_q", "score.gemm_cross_out", "score.gemm_ffn_up",
    "score.gemm_ffn_down", "score.self_attention", "score.cross_attention", "score.layernorm", "score.layernorm_score",
    "score.input_copy", "encode.gemm", "encode.causal_attention", "encode.layernorm", "encode.scatter_kv",
    "encode.gemm_cross_kv", "encode.global_pool"};

// Records a HIP event pair around each launch on the launching stream while
// enabled; totals are folded in when read.
constexpr size_t kProfileReserve = 2048;  // events made when profiling is enabled (1024 launches)
struct Profiler {
  bool on = false;
  uint64_t mask = ~0ull;  // classes recorded while on
  struct Rec {
    int cls;
    hipEvent_t a, b;
    double flops, bytes;
  };
  std::vector<hipEvent_t> spare;
  std::vector<Rec> recs;
  double ms[K_COUNT] = {}, flops[K_COUNT] = {}, bytes[K_COUNT] = {};
  int64_t n[K_COUNT] = {};
  hipEvent_t get() {
    if (!spare.empty()) {
      hipEvent_t e = spare.back();
      spare.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  // Event pairs are made ahead of time: an hipEventCreate while kernels run
  // can grow the runtime's signal pool, and that stalled the running kernel
  // by ~7 ms once per growth on MI355X (a 20-step run with every launch
  // bracketed had one step of 20.6 ms against a median of 13.3; with the
  // events made beforehand the slowest step was 13.7 ms).
  void reserve(size_t n) {
    while (spare.size() < n) {
      hipEvent_t e = nullptr;
      if (hipEventCreate(&e) != hipSuccess) return;
      spare.push_back(e);
    }
  }
  void clear() {
    for (auto& r : recs) {
      (void)hipEventSynchronize(r.b);
      spare.push_back(r.a);
      spare.push_back(r.b);
    }
    recs.clear();
    for (int k = 0; k < K_COUNT; ++k) ms[k] = flops[k] = bytes[k] = 0, n[k] = 0;
  }
  hipError_t fold() {
    for (auto& r : recs) {
      hipError_t e = hipEventSynchronize(r.b);
      if (e != hipSuccess) return e;
      float t = 0.f;
      e = hipEventElapsedTime(&t, r.a, r.b);
      if (e != hipSuccess) return e;
      ms[r.cls] += t;
      flops[r.cls] += r.flops;
      bytes[r.cls] += r.bytes;
      n[r.cls] += 1;
      spare.push_back(r.a);
      spare.push_back(r.b);
    }
    recs.clear();
    return hipSuccess;
  }
};
Profiler g_prof;

struct ProfScope {
  int cls;
  hipStream_t st;
  double fl, by;
  hipEvent_t a = nullptr;
  ProfScope(int c, hipStream_t s, double f, double b) : cls(c), st(s), fl(f), by(b) {
    if (g_prof.on && ((g_prof.mask >> c) & 1) && (a = g_prof.get())) (void)hipEventRecord(a, st);
  }
  ~ProfScope() {
    if (!a) return;
    hipEvent_t b = g_prof.get();
    if (!b) return;
    (void)hipEventRecord(b, st);
    g_prof.recs.push_back({cls, a, b, fl, by});
  }
};
}  // namespace

#define TX_LAUNCH(cls, fl, by, expr) \
  do {                               \
    ProfScope ps_((cls), st, (fl), (by)); \
    TX_HIP(expr);                    \
  } while (0)

extern "C" {

int tx_profile_enable(int32_t on) {
  g_prof.clear();
  g_prof.on = on != 0;
  g_prof.mask = ~0ull;
  if (g_prof.on) g_prof.reserve(kProfileReserve);
  return TX_OK;
}

int tx_profile_select(uint64_t class_mask) {
  g_prof.mask = class_mask;
  return TX_OK;
}

int32_t tx_profile_classes(void) { return K_COUNT; }

const char* tx_profile_class_name(int32_t i) { return (i >= 0 && i < K_COUNT) ? kClassNames[i] : ""; }

int tx_profile_read(double* total_ms, int64_t* launches, double* flops, double* bytes) {
  TX_HIP(g_prof.fold());
  for (int k = 0; k < K_COUNT; ++k) {
    if (total_ms) total_ms[k] = g_prof.ms[k];
    if (launches) launches[k] = g_prof.n[k];
    if (flops) flops[k] = g_prof.flops[k];
    if (bytes) bytes[k] = g_prof.bytes[k];
  }
  return TX_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ planning
namespace {

// Host-side metadata of one pass, uploaded in one copy to the workspace head.
struct Meta {
  std::vector<char> buf;
  template <class T>
  size_t put(const std::vector<T>& v) {
    const size_t o = align_up(buf.size());
    buf.resize(o + std::max<size_t>(v.size(), 1) * sizeof(T), 0);
    if (!v.empty()) memcpy(buf.data() + o, v.data(), v.size() * sizeof(T));
    return o;
  }
};

// kv-split of the pipelined cross-attention: partial slots per pass (each
// kXPartBytes of workspace).
constexpr int kXMaxParts = 512;

// Generous upper bound of a pass's metadata bytes.
size_t meta_bound(int n_req, int64_t rows, int64_t max_rows, int H) {
  const int64_t tiles = (int64_t)H * (rows / 32 + n_req + 1) + 8 * (max_rows / 32 + 2);
  const int64_t pool_chunks = rows / 64 + n_req + 1;
  const int64_t page_tiles = rows / kPage + n_req + 1;  // each request adds at most one partial page
  // cross-attention tiles (whole and split sets together), per-XCD offsets
  // and merges of both decoder layer kinds, with the alignment of their ten
  // arrays
  const int64_t xtiles = (int64_t)H * (rows / kXQueryBlock + n_req + 1) + kXMaxParts;  // per layer kind
  return align_up(8192 + (size_t)n_req * 160 + (size_t)tiles * sizeof(AttnTile) * 6 +
                  (size_t)pool_chunks * sizeof(PoolChunk) + (size_t)n_req * sizeof(PoolReq) +
                  (size_t)page_tiles * sizeof(ScatterTile) + 2 * (size_t)xtiles * sizeof(XTile) +
                  2 * (size_t)kXMaxParts * sizeof(XMerge) + 4 * 9 * sizeof(int32_t) + 10 * 256);
}

// Resident blocks of the cross-attention on the current device (kXBlocksPerCu
// per CU), the CU count looked up once per device.
int xattn_resident_blocks() {
  static std::atomic<int> cu_of_device[64];
  int dev = 0, n_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = -1;
  if (dev >= 0) n_cu = cu_of_device[dev].load(std::memory_order_relaxed);
  if (n_cu <= 0) {
    if (dev < 0 || hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 8)
      n_cu = 256;
    if (dev >= 0) cu_of_device[dev].store(n_cu, std::memory_order_relaxed);
  }
  return n_cu / 8 * 8 * kXBlocksPerCu;
}

// Attention worklist: tiles of q_block queries for every (request, head),
// longest groups first, each (request, head) group kept on one XCD (the
// hardware deals block b to XCD b % 8, so group g's tiles sit at indices
// congruent to its XCD) and XCDs balanced by total cost.
struct Group {
  int req, head, nq;
  int64_t cost;
};
void attn_tiles(const std::vector<AttnReq>& reqs, int H, int q_block, bool causal, std::vector<AttnTile>& out) {
  out.clear();
  std::vector<Group> groups;
  for (int r = 0; r < (int)reqs.size(); ++r) {
    const int nq = reqs[r].qa_n + reqs[r].qb_n;
    if (nq <= 0) continue;
    int64_t cost = 0;
    for (int q0 = 0; q0 < nq; q0 += q_block) {
      const int qn = std::min(q_block, nq - q0);
      const int64_t keys = causal ? std::min<int64_t>(reqs[r].kv_len, reqs[r].pos0 + q0 + qn) : reqs[r].kv_len;
      cost += (int64_t)q_block * ((keys + kPage - 1) / kPage) + 4;
    }
    for (int h = 0; h < H; ++h) groups.push_back({r, h, nq, cost});
  }
  std::stable_sort(groups.begin(), groups.end(), [](const Group& a, const Group& b) { return a.cost > b.cost; });
  std::vector<AttnTile> lists[8];
  int64_t load[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (const Group& g : groups) {
    int x = 0;
    for (int k = 1; k < 8; ++k)
      if (load[k] < load[x]) x = k;
    load[x] += g.cost;
    for (int q0 = 0; q0 < g.nq; q0 += q_block) lists[x].push_back({g.req, g.head, q0, std::min(q_block, g.nq - q0)});
  }
  size_t longest = 0;
  for (auto& l : lists) longest = std::max(longest, l.size());
  out.assign(longest * 8, AttnTile{0, 0, 0, 0});
  for (int x = 0; x < 8; ++x)
    for (size_t s = 0; s < lists[x].size(); ++s) out[s * 8 + x] = lists[x][s];
}

void self_tiles(const std::vector<SelfReq>& reqs, int H, int q_block, bool cand_only, std::vector<SelfTile>& out) {
  out.clear();
  for (int r = 0; r < (int)reqs.size(); ++r) {
    const int nq = cand_only ? reqs[r].C : reqs[r].S + reqs[r].C;
    for (int h = 0; h < H; ++h)
      for (int q0 = 0; q0 < nq; q0 += q_block) out.push_back({r, h, q0, std::min(q_block, nq - q0)});
  }
}

int check_offsets(const int64_t* o, int n, const char* what, int64_t min_count) {
  if (!o) return fail(TX_E_INVALID, "%s offsets are null", what);
  if (o[0] < 0) return fail(TX_E_INVALID, "%s offsets[0] = %lld", what, (long long)o[0]);
  for (int i = 0; i < n; ++i) {
    if (o[i + 1] < o[i]) return fail(TX_E_INVALID, "%s offsets decrease at %d", what, i);
    if (o[i + 1] - o[i] < min_count)
      return fail(TX_E_INVALID, "%s count %lld of request %d below %lld", what, (long long)(o[i + 1] - o[i]), i,
                  (long long)min_count);
    if (o[i + 1] - o[i] > INT32_MAX / 4) return fail(TX_E_INVALID, "%s count too large", what);
  }
  if (o[n] > INT32_MAX) return fail(TX_E_INVALID, "%s offsets exceed 2^31 rows", what);
  return TX_OK;
}

int check_ids(const tx_kv_cache* c, int n, const int32_t* ids) {
  if (n > 0 && !ids) return fail(TX_E_INVALID, "request ids are null");
  std::vector<char> seen(c->max_req, 0);
  for (int i = 0; i < n; ++i) {
    if (ids[i] < 0 || ids[i] >= c->max_req) return fail(TX_E_INVALID, "request id %d out of range", ids[i]);
    if (seen[ids[i]]) return fail(TX_E_INVALID, "request id %d repeated", ids[i]);
    seen[ids[i]] = 1;
  }
  return TX_OK;
}

// Per-row activation bytes of each operation: the model-type buffers, two
// pre-LN sum buffers (the sum type has the model type's width) and two
// LayerNorm row-statistics records.
size_t row_bytes(const tx_model* m, int op) {
  const size_t d = m->d, F = m->F;
  if (op == TX_OP_SCORE) return m->esz * (d + 3 * d + d + d + 2 * d + F) + 2 * sizeof(LnRow);
  return m->esz * (d + 3 * d + d + 2 * d + std::max(F, (size_t)(2 * m->n_dec) * d)) + 2 * sizeof(LnRow);
}

// Workspace of the global-token pooling in an encoder pass: chunk partial
// states, the pooled tokens and their cross K/V rows.
size_t pool_pass_bytes(const tx_model* m, int op, int n, int64_t rows) {
  if (!m->gpool || op == TX_OP_SCORE) return 0;
  const size_t d = m->d;
  return align_up((size_t)(rows / 64 + n + 1) * (d + 2) * 4) + align_up((size_t)n * d * m->esz) +
         align_up((size_t)n * 2 * m->n_dec * d * m->esz) + 3 * 256;
}

// The dense bf16 d_h = 128 decoder cross-attention runs on the tile list of
// xattn_plan (with kv-split); its partial slots take a fixed workspace area.
bool xattn_pipe_used(const tx_model* m) { return m->l_local == 0 && cross_attention_split_ok(m->bf, m->dh); }
size_t xattn_part_area(const tx_model* m, int op) {
  return op == TX_OP_SCORE && xattn_pipe_used(m) ? align_up((size_t)kXMaxParts * kXPartBytes) : 0;
}

size_t pass_bytes(const tx_model* m, int op, int n, int64_t rows, int64_t max_rows) {
  return meta_bound(n, rows, max_rows, m->H) + align_up(rows * row_bytes(m, op)) + 11 * 256 +
         pool_pass_bytes(m, op, n, rows) + xattn_part_area(m, op);
}

// rows of request i for the op
int64_t req_rows(int op, int i, const int64_t* a, const int64_t* b) {
  return (a[i + 1] - a[i]) + (op == TX_OP_SCORE ? (b[i + 1] - b[i]) : 0);
}

// Split requests into consecutive groups that fit the workspace.
// meta_cap bounds each pass's metadata (the uploads of the no-allocation
// entry point go through fixed pinned staging).
int plan_passes(const tx_model* m, int op, int n, const int64_t* a, const int64_t* b, size_t ws_bytes,
                std::vector<int>& cuts, size_t meta_cap = SIZE_MAX) {
  cuts.assign(1, 0);
  int start = 0;
  int64_t rows = 0, mx = 0;
  for (int i = 0; i < n; ++i) {
    const int64_t r = req_rows(op, i, a, b);
    if (pass_bytes(m, op, 1, r, r) > ws_bytes)
      return fail(TX_E_NOMEM, "workspace %zu bytes cannot hold request %d (%zu needed)", ws_bytes, i,
                  pass_bytes(m, op, 1, r, r));
    if (meta_bound(1, r, r, m->H) > meta_cap)
      return fail(TX_E_NOMEM, "request %d: pass metadata above the %zu bytes of fixed staging", i, meta_cap);
    if (i > start && (pass_bytes(m, op, i - start + 1, rows + r, std::max(mx, r)) > ws_bytes ||
                      meta_bound(i - start + 1, rows + r, std::max(mx, r), m->H) > meta_cap)) {
      cuts.push_back(i);
      start = i;
      rows = 0;
      mx = 0;
    }
    rows += r;
    mx = std::max(mx, r);
  }
  if (cuts.back() != n) cuts.push_back(n);
  return TX_OK;
}

struct Acts {
  char *T, *QKV, *A, *O, *Y, *Hf;
};

}  // namespace

extern "C" {

size_t tx_workspace_bytes(const tx_kv_cache* c, int32_t op, int32_t n, const int64_t* a, const int64_t* b) {
  if (!c || n < 0 || !a || (op == TX_OP_SCORE && !b) || op < 0 || op > 2) return 0;
  int64_t rows = 0, mx = 0;
  for (int i = 0; i < n; ++i) {
    const int64_t r = req_rows(op, i, a, b);
    rows += r;
    mx = std::max(mx, r);
  }
  return pass_bytes(c->m, op, n, rows, mx);
}

size_t tx_workspace_min_bytes(const tx_kv_cache* c, int32_t op, int32_t n, const int64_t* a, const int64_t* b) {
  if (!c || n < 0 || !a || (op == TX_OP_SCORE && !b) || op < 0 || op > 2) return 0;
  size_t best = 0;
  for (int i = 0; i < n; ++i) {
    const int64_t r = req_rows(op, i, a, b);
    best = std::max(best, pass_bytes(c->m, op, 1, r, r));
  }
  return best;
}

}  // extern "C"

// ------------------------------------------------------------------ encoder passes
namespace {

// Encoder layers over the rows of one pass (whole sequences for build, new
// events for append), then the cross-attention K/V of every decoder layer.
// reqs[i]: rows row0.. of request slot, positions pos0.., kv_len = pos0 + n.
int run_encoder_pass(tx_kv_cache* c, const char* X, int64_t rows, const std::vector<ScatterReq>& sreqs, char* ws,
                     hipStream_t st) {
  const tx_model* m = c->m;
  const bool bf = m->bf;
  const int d = m->d, F = m->F, n = (int)sreqs.size();
  std::vector<AttnReq> areqs(n);
  int64_t mx = 0;
  for (int i = 0; i < n; ++i) {
    const ScatterReq& s = sreqs[i];
    areqs[i] = AttnReq{s.row0, s.n, 0, 0, s.pos0 + s.n, s.pos0, s.slot, 0};
    mx = std::max<int64_t>(mx, s.n);
  }
  // a few new tokens per request (an append): one wave per (request, head)
  // streams the cached pages through registers
  const int qb = (mx <= kDecodeQBlock && paged_attention_decode_ok(bf, m->dh, m->R)) ? kDecodeQBlock
                                                                                 : paged_attention_q_block(bf, m->dh);
  std::vector<AttnTile> tiles;
  attn_tiles(areqs, m->H, qb, true, tiles);
  // global-token pooling: 64-row chunks of each request's new rows
  std::vector<PoolChunk> chunks;
  std::vector<PoolReq> preqs;
  if (m->gpool) {
    for (int i = 0; i < n; ++i) {
      const ScatterReq& s = sreqs[i];
      const int c0 = (int)chunks.size();
      for (int r = 0; r < s.n; r += 64) chunks.push_back({i, s.row0 + r, std::min(64, s.n - r), 0});
      preqs.push_back({c0, (int)chunks.size() - c0, s.slot, s.pos0 == 0 ? 1 : 0});
    }
  }
  // cache pages written by this pass, split per request
  std::vector<ScatterTile> ptiles;
  for (const ScatterReq& s : sreqs)
    for (int p = s.pos0 / kPage; p * kPage < s.pos0 + s.n; ++p) {
      const int t0 = std::max(s.pos0, p * kPage) - p * kPage, t1 = std::min(s.pos0 + s.n, (p + 1) * kPage) - p * kPage;
      ptiles.push_back(ScatterTile{s.slot, p, t0, t1, s.row0 + (p * kPage + t0 - s.pos0)});
    }
  Meta meta;
  const size_t o_areq = meta.put(areqs), o_tiles = meta.put(tiles);
  const size_t o_chunks = meta.put(chunks), o_preqs = meta.put(preqs), o_ptiles = meta.put(ptiles);
  const size_t mb = meta_bound(n, rows, mx, m->H);
  if (meta.buf.size() > mb) return fail(TX_E_NOMEM, "internal: metadata %zu > bound %zu", meta.buf.size(), mb);
  TX_HIP(c->st.upload(ws, meta.buf.data(), meta.buf.size(), st));
  const ScatterTile* d_ptiles = (const ScatterTile*)(ws + o_ptiles);
  const int n_ptiles = (int)ptiles.size();
  const AttnReq* d_areq = (const AttnReq*)(ws + o_areq);
  const AttnTile* d_tiles = (const AttnTile*)(ws + o_tiles);
  Carver cv(ws + mb);
  const size_t es = m->esz;
  char* T = cv.take<char*>(rows * d * es);
  char* QKV = cv.take<char*>(rows * 3 * d * es);
  char* A = cv.take<char*>(rows * d * es);
  // pre-LN sums and LayerNorm row statistics, alternating between sublayers:
  // sublayer k writes Ys[k % 2] and adds LN(Ys[(k - 1) % 2]) as its residual
  char* Ys[2] = {cv.take<char*>(rows * d * es), cv.take<char*>(rows * d * es)};
  LnRow* Ss[2] = {cv.take<LnRow*>(rows * sizeof(LnRow)), cv.take<LnRow*>(rows * sizeof(LnRow))};
  char* Hf = cv.take<char*>(rows * std::max(F, 2 * m->n_dec * d) * es);
  float* pool_part = nullptr;
  char *gtok = nullptr, *gkv_rows = nullptr;
  if (m->gpool) {
    pool_part = cv.take<float*>(chunks.size() * (size_t)(d + 2) * 4);
    gtok = cv.take<char*>((size_t)n * d * es);
    gkv_rows = cv.take<char*>((size_t)n * 2 * m->n_dec * d * es);
  }
  const int M = (int)rows;
  const double dd = d, Md = (double)M, esd = (double)es;
  double attn_pairs = 0.0, kv_bytes = 0.0;
  for (const AttnReq& r : areqs) {
    attn_pairs += (double)r.qa_n * r.pos0 + 0.5 * (double)r.qa_n * (r.qa_n + 1);
    kv_bytes += (double)r.kv_len * 2 * d * es;
  }
  auto gemm_fb = [&](double N, double K) { return std::make_pair(2 * Md * N * K, esd * (Md * K + N * K + Md * N)); };
  const float eps = m->cfg.ln_eps;
  for (int e = 0; e < m->n_enc; ++e) {
    const EncLayer& L = m->enc[e];
    const char* in = e == 0 ? X : T;
    char *Y0 = Ys[0], *Y1 = Ys[1];  // sublayers 2e (attention) and 2e + 1 (FFN)
    LnRow *S0 = Ss[0], *S1 = Ss[1];
    auto g1 = gemm_fb(3 * dd, dd), g2 = gemm_fb(dd, dd), g3 = gemm_fb(F, dd), g4 = gemm_fb(dd, F);
    TX_LAUNCH(K_ENC_GEMM, g1.first, g1.second,
              launch_gemm(bf, in, d, L.qkv.w, L.qkv.b, nullptr, 0, QKV, 3 * d, M, 3 * d, d, EPI_BIAS, st));
    TX_LAUNCH(K_SCATTER, 0, 4 * Md * dd * esd,
              launch_scatter_kv(bf, QKV + d * es, 3 * d, 1, e, c->pool, c->d_table, c->max_pages, c->geom, d_ptiles,
                                n_ptiles, st));
    TX_LAUNCH(K_ENC_ATTN, 4 * dd * attn_pairs, kv_bytes + 2 * Md * dd * esd,
              launch_paged_attention(bf, QKV, 3 * d, A, d, c->pool, c->d_table, c->max_pages, c->geom, e, d_areq,
                                     d_tiles, (int)tiles.size(), true, L.rel, m->R, qb, st));
    // residual: the input tokens (first layer) or the previous layer's output
    // LN2(Y1), recomputed from its pre-LN sum
    TX_LAUNCH(K_ENC_GEMM, g2.first, g2.second + Md * dd * esd,
              e == 0 ? launch_gemm(bf, A, d, L.o.w, L.o.b, X, d, Y0, d, M, d, d, EPI_BIAS_RESID, st)
                     : launch_gemm(bf, A, d, L.o.w, L.o.b, Y1, d, Y0, d, M, d, d, EPI_BIAS_RESLN, st,
                                   LnResid{S1, m->enc[e - 1].ln2g, m->enc[e - 1].ln2b}));
    TX_LAUNCH(K_ENC_LAYERNORM, 0, 2 * Md * dd * esd, launch_layernorm(bf, Y0, T, S0, L.ln1g, L.ln1b, M, d, eps, st));
    TX_LAUNCH(K_ENC_GEMM, g3.first, g3.second,
              launch_gemm(bf, T, d, L.f1.w, L.f1.b, nullptr, 0, Hf, F, M, F, d, EPI_BIAS_GELU, st));
    TX_LAUNCH(K_ENC_GEMM, g4.first, g4.second + Md * dd * esd,
              launch_gemm(bf, Hf, F, L.f2.w, L.f2.b, Y0, d, Y1, d, M, d, F, EPI_BIAS_RESLN, st,
                          LnResid{S0, L.ln1g, L.ln1b}));
    TX_LAUNCH(K_ENC_LAYERNORM, 0, 2 * Md * dd * esd, launch_layernorm(bf, Y1, T, S1, L.ln2g, L.ln2b, M, d, eps, st));
  }
  const int nkv = 2 * d * m->n_dec;
  auto g5 = gemm_fb(nkv, dd);
  TX_LAUNCH(K_XKV_GEMM, g5.first, g5.second,
            launch_gemm(bf, T, d, m->xkv.w, m->xkv.b, nullptr, 0, Hf, nkv, M, nkv, d, EPI_BIAS, st));
  TX_LAUNCH(K_SCATTER, 0, 2 * Md * nkv * esd,
            launch_scatter_kv(bf, Hf, nkv, m->n_dec, m->n_enc, c->pool, c->d_table, c->max_pages, c->geom, d_ptiles,
                              n_ptiles, st));
  if (m->gpool) {
    // fold the new rows into each request's pooling state, then project the
    // pooled token with every decoder layer's cross K/V weights
    const PoolReq* d_preqs = (const PoolReq*)(ws + o_preqs);
    const double nd = n;
    TX_LAUNCH(K_POOL, 4 * Md * dd, 2 * Md * dd * esd,
              launch_pool(bf, T, d, m->wpool, 1.f / sqrtf((float)d), (const PoolChunk*)(ws + o_chunks),
                          (int)chunks.size(), d_preqs, n, pool_part, c->d_pool_ml, c->d_pool_acc, gtok, st));
    TX_LAUNCH(K_POOL, 2 * nd * nkv * dd, esd * (nd * dd + nkv * dd + nd * nkv),
              launch_gemm(bf, gtok, d, m->xkv.w, m->xkv.b, nullptr, 0, gkv_rows, nkv, n, nkv, d, EPI_BIAS, st));
    TX_LAUNCH(K_POOL, 0, 2 * nd * nkv * esd, launch_store_rows(bf, gkv_rows, nkv, d_preqs, n, c->d_gkv, st));
  }
  return TX_OK;
}

int encode_call(tx_kv_cache* c, int op, int n, const int32_t* ids, const void* X, const int64_t* off, void* ws,
                size_t ws_bytes, hipStream_t st) {
  std::vector<int> cuts;
  TX_CHECK(plan_passes(c->m, op, n, off, nullptr, ws_bytes, cuts));
  const size_t es = c->m->esz;
  const int d = c->m->d;
  for (size_t p = 0; p + 1 < cuts.size(); ++p) {
    const int a = cuts[p], b = cuts[p + 1];
    std::vector<ScatterReq> sreqs;
    for (int i = a; i < b; ++i) {
      const int64_t cnt = off[i + 1] - off[i];
      const int64_t pos0 = op == TX_OP_BUILD ? 0 : c->len[ids[i]];
      sreqs.push_back({(int32_t)(off[i] - off[a]), (int32_t)cnt, (int32_t)pos0, ids[i]});
    }
    const char* X0 = (const char*)X + (size_t)off[a] * d * es;
    TX_CHECK(run_encoder_pass(c, X0, off[b] - off[a], sreqs, (char*)ws, st));
  }
  return TX_OK;
}

int common_checks(const tx_kv_cache* c, int n, const int32_t* ids, const void* ws) {
  if (!c) return fail(TX_E_INVALID, "cache is null");
  if (n < 0) return fail(TX_E_INVALID, "n_req %d", n);
  TX_CHECK(check_ids(c, n, ids));
  if (((uintptr_t)ws & 255)) return fail(TX_E_INVALID, "workspace not 256-byte aligned");
  return TX_OK;
}

int check_weights(const tx_kv_cache* c) {
  if (!c->m->weights_set) return fail(TX_E_INVALID, "model weights have not been set");
  return TX_OK;
}

int check_tokens(const tx_kv_cache* c, int n, const void* X, const int64_t* off, const char* what) {
  if (off[n] > off[0] && !X) return fail(TX_E_INVALID, "%s pointer is null", what);
  if (((uintptr_t)X % c->m->esz)) return fail(TX_E_INVALID, "%s pointer misaligned", what);
  return TX_OK;
}

}  // namespace

extern "C" {

int kv_cache_build(tx_kv_cache* c, int32_t n, const int32_t* ids, const void* X, const int64_t* off, void* ws,
                   size_t ws_bytes, hipStream_t st) {
  TX_CHECK(common_checks(c, n, ids, ws));
  if (n == 0) return TX_OK;
  TX_CHECK(check_offsets(off, n, "behavior", 1));
  TX_CHECK(check_tokens(c, n, X, off, "behavior"));
  for (int i = 0; i < n; ++i)
    if (off[i + 1] - off[i] > c->max_tokens)
      return fail(TX_E_INVALID, "request %d: L = %lld exceeds max_tokens %lld", ids[i],
                  (long long)(off[i + 1] - off[i]), (long long)c->max_tokens);
  std::vector<int> cuts;
  TX_CHECK(plan_passes(c->m, TX_OP_BUILD, n, off, nullptr, ws_bytes, cuts));
  if (!ws) return fail(TX_E_INVALID, "workspace is null");
  int64_t need = 0, freed = 0;
  for (int i = 0; i < n; ++i) {
    need += (off[i + 1] - off[i] + kPage - 1) / kPage;
    freed += (int64_t)c->pages[ids[i]].size();
  }
  if (need > (int64_t)c->free_list.size() + freed)
    return fail(TX_E_NOMEM, "page pool exhausted: need %lld pages, %lld free", (long long)need,
                (long long)(c->free_list.size() + freed));
  TX_CHECK(check_weights(c));
  // commit page assignment
  for (int i = 0; i < n; ++i) {
    auto& pg = c->pages[ids[i]];
    for (int32_t p : pg) c->free_list.push_back(p);
    pg.clear();
  }
  for (int i = 0; i < n; ++i) {
    const int64_t np = (off[i + 1] - off[i] + kPage - 1) / kPage;
    auto& pg = c->pages[ids[i]];
    for (int64_t k = 0; k < np; ++k) {
      pg.push_back(c->free_list.back());
      c->free_list.pop_back();
      c->h_table[(size_t)ids[i] * c->max_pages + k] = pg.back();
    }
  }
  // from here on a failure leaves these requests without a cache, holding
  // their pages until release
  int rc = TX_OK;
  const hipError_t e = c->st.upload(c->d_table, c->h_table.data(), c->h_table.size() * 4, st);
  if (e != hipSuccess) rc = fail(TX_E_HIP, "page table upload failed: %s", hipGetErrorString(e));
  if (rc == TX_OK) rc = encode_call(c, TX_OP_BUILD, n, ids, X, off, ws, ws_bytes, st);
  for (int i = 0; i < n; ++i) c->len[ids[i]] = rc == TX_OK ? off[i + 1] - off[i] : -1;
  return rc;
}

int kv_cache_append(tx_kv_cache* c, int32_t n, const int32_t* ids, const void* X, const int64_t* off, void* ws,
                    size_t ws_bytes, hipStream_t st) {
  TX_CHECK(common_checks(c, n, ids, ws));
  if (n == 0) return TX_OK;
  TX_CHECK(check_offsets(off, n, "event", 1));
  TX_CHECK(check_tokens(c, n, X, off, "event"));
  for (int i = 0; i < n; ++i) {
    if (c->len[ids[i]] < 0) return fail(TX_E_NOCACHE, "request %d has no cache", ids[i]);
    if (c->len[ids[i]] + (off[i + 1] - off[i]) > c->max_tokens)
      return fail(TX_E_INVALID, "request %d would exceed max_tokens", ids[i]);
  }
  std::vector<int> cuts;
  TX_CHECK(plan_passes(c->m, TX_OP_APPEND, n, off, nullptr, ws_bytes, cuts));
  if (!ws) return fail(TX_E_INVALID, "workspace is null");
  int64_t need = 0;
  for (int i = 0; i < n; ++i) {
    const int64_t L1 = c->len[ids[i]] + off[i + 1] - off[i];
    need += (L1 + kPage - 1) / kPage - (int64_t)c->pages[ids[i]].size();
  }
  if (need > (int64_t)c->free_list.size())
    return fail(TX_E_NOMEM, "page pool exhausted: need %lld pages, %zu free", (long long)need, c->free_list.size());
  TX_CHECK(check_weights(c));
  for (int i = 0; i < n; ++i) {
    const int64_t L1 = c->len[ids[i]] + off[i + 1] - off[i];
    auto& pg = c->pages[ids[i]];
    while ((int64_t)pg.size() * kPage < L1) {
      pg.push_back(c->free_list.back());
      c->free_list.pop_back();
      c->h_table[(size_t)ids[i] * c->max_pages + pg.size() - 1] = pg.back();
    }
  }
  // from here on a failure leaves these requests without a cache, holding
  // their pages until release
  int rc = TX_OK;
  const hipError_t e = c->st.upload(c->d_table, c->h_table.data(), c->h_table.size() * 4, st);
  if (e != hipSuccess) rc = fail(TX_E_HIP, "page table upload failed: %s", hipGetErrorString(e));
  if (rc == TX_OK) rc = encode_call(c, TX_OP_APPEND, n, ids, X, off, ws, ws_bytes, st);
  for (int i = 0; i < n; ++i) c->len[ids[i]] = rc == TX_OK ? c->len[ids[i]] + off[i + 1] - off[i] : -1;
  return rc;
}

}  // extern "C"

// ------------------------------------------------------------------ score
namespace {

// Decoder + head over groups a .. b-1 (a group = one serving event: its
// serving and candidate rows, decoded against the first kvlen[r] cached
// tokens of request ids[r]).
int run_score_pass(const tx_kv_cache* c, const int32_t* ids, const int64_t* kvlen, int a, int b, const char* xs,
                   const int64_t* so, const char* xc, const int64_t* co, float* scores, char* ws, hipStream_t st,
                   bool fixed_staging) {
  const tx_model* m = c->m;
  const bool bf = m->bf;
  const int d = m->d, F = m->F, H = m->H;
  const size_t es = m->esz;
  const int64_t Ms = so[b] - so[a], Mc = co[b] - co[a], M64 = Ms + Mc;
  if (Mc == 0) return TX_OK;
  const int M = (int)M64;
  const int n = b - a;
  std::vector<SelfReq> sreq(n);
  std::vector<AttnReq> full(n), cand(n);
  int64_t mx = 0;
  for (int i = 0; i < n; ++i) {
    const int r = a + i;
    const int S = (int)(so[r + 1] - so[r]), C = (int)(co[r + 1] - co[r]);
    const int s_row = (int)(so[r] - so[a]), c_row = (int)(Ms + co[r] - co[a]);
    const int kv = (int)kvlen[r];
    sreq[i] = SelfReq{s_row, S, c_row, C};
    full[i] = AttnReq{s_row, S, c_row, C, kv, 0, ids[r], 0};
    cand[i] = AttnReq{c_row, C, 0, 0, kv, 0, ids[r], 0};
    mx = std::max<int64_t>(mx, S + C);
  }
  const bool sparse = m->l_local > 0;
  const int qb =
      sparse ? lg_attention_q_block(bf, m->l_local, m->gpool, H, m->dh) : paged_attention_q_block(bf, m->dh);
  // head groups of the tile plan: a sparse MFMA tile serves several heads
  const int th = sparse ? H / lg_attention_heads_per_tile(bf, m->l_local, m->gpool, H, m->dh) : H;
  const int sqb = self_attention_q_block(bf, m->dh);
  std::vector<AttnTile> t_full, t_cand;
  std::vector<SelfTile> s_full, s_cand;
  const bool xpipe = xattn_pipe_used(m);
  const int xblocks = xpipe ? xattn_resident_blocks() : 0;
  XPlan x_full, x_cand;
  if (m->n_dec > 1) {
    if (xpipe) xattn_plan(full, H, xblocks, kXMaxParts, x_full);
    else attn_tiles(full, th, qb, false, t_full);
    self_tiles(sreq, H, sqb, false, s_full);
  }
  if (xpipe) xattn_plan(cand, H, xblocks, kXMaxParts, x_cand);
  else attn_tiles(cand, th, qb, false, t_cand);
  self_tiles(sreq, H, sqb, true, s_cand);
  Meta meta;
  const size_t o_sreq = meta.put(sreq), o_full = meta.put(full), o_cand = meta.put(cand);
  const size_t o_tf = meta.put(t_full), o_tc = meta.put(t_cand), o_sf = meta.put(s_full), o_sc = meta.put(s_cand);
  // cross-attention tile sets on the device: whole-request tiles, their
  // per-XCD offsets, kv-split tiles, theirs, and the merge items
  struct XDev {
    size_t wt, wo, st, so, mg;
  };
  auto put_plan = [&](const XPlan& xp) {
    return XDev{meta.put(xp.whole.tiles), meta.put(xp.whole.xoff), meta.put(xp.split.tiles), meta.put(xp.split.xoff),
                meta.put(xp.merges)};
  };
  const XDev xd_full = put_plan(x_full), xd_cand = put_plan(x_cand);
  const size_t mb = meta_bound(n, M64, mx, H);
  if (meta.buf.size() > mb) return fail(TX_E_NOMEM, "internal: metadata %zu > bound %zu", meta.buf.size(), mb);
  TX_HIP(c->st.upload(ws, meta.buf.data(), meta.buf.size(), st, !fixed_staging));
  Carver cv(ws + mb);
  char* T = cv.take<char*>(M64 * d * es);
  char* QKV = cv.take<char*>(M64 * 3 * d * es);
  char* A = cv.take<char*>(M64 * d * es);
  char* O = cv.take<char*>(M64 * d * es);
  // pre-LN sums and LayerNorm row statistics, alternating between sublayers:
  // sublayer k writes Ys[k % 2] and adds LN(Ys[(k - 1) % 2]) as its residual
  char* Ys[2] = {cv.take<char*>(M64 * d * es), cv.take<char*>(M64 * d * es)};
  LnRow* Ss[2] = {cv.take<LnRow*>(M64 * sizeof(LnRow)), cv.take<LnRow*>(M64 * sizeof(LnRow))};
  char* Hf = cv.take<char*>(M64 * F * es);
  float* xpart = xpipe ? cv.take<float*>(kXMaxParts * kXPartBytes) : nullptr;
  // The first layer reads the serving and candidate tokens where they are
  // (its QKV GEMM and the self-attention output GEMM's residual run once per
  // token array) when the bf16 GEMMs can take them (16-byte aligned rows) and
  // both arrays fill the GPU on their own (8192 rows or more: 32 row tiles
  // of the persistent GEMM); otherwise they are copied into T, where the
  // later layers' input lives.
  const char* Xs = xs + (size_t)so[a] * d * es;
  const char* Xc = xc + (size_t)co[a] * d * es;
  const bool direct = (Ms == 0 || Ms >= 8192) && Mc >= 8192 &&
                      (!bf || ((Ms == 0 || (uintptr_t)Xs % 16 == 0) && (uintptr_t)Xc % 16 == 0 &&
                               ((size_t)d * es) % 16 == 0));
  if (!direct)
    TX_LAUNCH(K_COPY, 0, 2.0 * M64 * d * es, [&]() -> hipError_t {
      if (Ms) {
        hipError_t e = hipMemcpyAsync(T, Xs, (size_t)Ms * d * es, hipMemcpyDeviceToDevice, st);
        if (e != hipSuccess) return e;
      }
      return hipMemcpyAsync(T + (size_t)Ms * d * es, Xc, (size_t)Mc * d * es, hipMemcpyDeviceToDevice, st);
    }());
  const float eps = m->cfg.ln_eps;
  const double dd = d, esd = (double)es;
  // algorithmic work of the attention launches: (query, key) pairs and cache bytes
  double pairs_full = 0, pairs_cand = 0, self_full = 0, self_cand = 0, kvb = 0;
  for (int i = 0; i < n; ++i) {
    const double S = sreq[i].S, C = sreq[i].C;
    // keys per query: the whole cache, or the sparse set
    const double kv = sparse ? std::min(full[i].kv_len, m->l_local) + (m->gpool ? 1 : 0) : full[i].kv_len;
    pairs_full += (S + C) * kv;
    pairs_cand += C * kv;
    self_full += 0.5 * S * (S + 1) + C * (S + 1);
    self_cand += C * (S + 1);
    kvb += kv * 2 * dd * esd;
  }
  for (int l = 0; l < m->n_dec; ++l) {
    const DecLayer& L = m->dec[l];
    const bool last = l == m->n_dec - 1;
    const XPlan& xp = last ? x_cand : x_full;
    const XDev& xd = last ? xd_cand : xd_full;
    // rows from r0 on continue past the self-attention: all rows, or only the
    // candidates in the last layer (serving rows there only supply keys/values)
    const int r0 = last ? (int)Ms : 0, Mr = M - r0;
    const double Mrd = Mr, Md = M;
    const size_t ro = (size_t)r0 * d * es;
    const AttnReq* areq = (const AttnReq*)(ws + (last ? o_cand : o_full));
    const AttnTile* at = (const AttnTile*)(ws + (last ? o_tc : o_tf));
    const int n_at = (int)(last ? t_cand.size() : t_full.size());
    const SelfTile* stl = (const SelfTile*)(ws + (last ? o_sc : o_sf));
    const int n_st = (int)(last ? s_cand.size() : s_full.size());
    auto gf = [&](double rows, double N, double K, double extra) {
      return std::make_pair(2 * rows * N * K, esd * (rows * K + N * K + rows * N * (1 + extra)));
    };
    auto q = gf(Md, 3 * dd, dd, 0), o = gf(Mrd, dd, dd, 1), xq = gf(Mrd, dd, dd, 0), xo = gf(Mrd, dd, dd, 1),
         f1 = gf(Mrd, F, dd, 0), f2 = gf(Mrd, dd, F, 1);
    // sublayers 3l (self-attention), 3l + 1 (cross-attention), 3l + 2 (FFN):
    // pre-LN sum buffer and row statistics of sublayer k, rows from r0 on
    auto Yk = [&](int k) { return Ys[k & 1] + ro; };
    auto Sk = [&](int k) { return Ss[k & 1] + r0; };
    const int k0 = 3 * l;
    // LayerNorm folds (bf16): the LayerNorms before the cross-Q and FFN-up
    // GEMMs (rows r0 ..) and before the next layer's QKV GEMM (all rows) write
    // only their row statistics, and those GEMMs multiply the stored pre-LN
    // sums by the gain-scaled weights (EPI_LN); T is then not written at all
    // (a model-level choice: a score does not depend on the batch it is in)
    const bool fold = m->ln_fold && gemm_ln_ok(d, d, d, d) && gemm_ln_ok(F, d, d, F);
    const bool fold_qkv = m->ln_fold && gemm_ln_ok(3 * d, d, d, 3 * d);
    const bool fold_in = l > 0 && fold_qkv, fold_out = !last && fold_qkv;
    // layer input rows r0 .. M - 1: T, or the token arrays in place (first layer)
    const bool in_place = l == 0 && direct;
    TX_LAUNCH(K_GEMM_QKV, q.first, q.second, [&]() -> hipError_t {
      if (fold_in)
        return launch_gemm(bf, Ys[(k0 - 1) & 1], d, L.qkvf.w, L.qkvf.b, nullptr, 0, QKV, 3 * d, M, 3 * d, d, EPI_LN,
                           st, LnResid{Ss[(k0 - 1) & 1], L.qkvf.cs, nullptr});
      if (!in_place) return launch_gemm(bf, T, d, L.qkv.w, L.qkv.b, nullptr, 0, QKV, 3 * d, M, 3 * d, d, EPI_BIAS, st);
      hipError_t e = launch_gemm(bf, Xs, d, L.qkv.w, L.qkv.b, nullptr, 0, QKV, 3 * d, (int)Ms, 3 * d, d, EPI_BIAS, st);
      if (e != hipSuccess) return e;
      return launch_gemm(bf, Xc, d, L.qkv.w, L.qkv.b, nullptr, 0, QKV + (size_t)Ms * 3 * d * es, 3 * d, (int)Mc,
                         3 * d, d, EPI_BIAS, st);
    }());
    TX_LAUNCH(K_SELF_ATTN, 4 * dd * (last ? self_cand : self_full), esd * (3 * Md * dd + Mrd * dd),
              launch_self_attention(bf, QKV, d, H, A, (const SelfReq*)(ws + o_sreq), stl, n_st, last, st));
    // residual: the layer input, i.e. the tokens (first layer) or the previous
    // layer's output LN3, recomputed from its pre-LN sum
    TX_LAUNCH(K_GEMM_O, o.first, o.second, [&]() -> hipError_t {
      if (l > 0)
        return launch_gemm(bf, A + ro, d, L.o.w, L.o.b, Yk(k0 - 1), d, Yk(k0), d, Mr, d, d, EPI_BIAS_RESLN, st,
                           LnResid{Sk(k0 - 1), m->dec[l - 1].ln3g, m->dec[l - 1].ln3b});
      if (!in_place)
        return launch_gemm(bf, A + ro, d, L.o.w, L.o.b, T + ro, d, Yk(k0), d, Mr, d, d, EPI_BIAS_RESID, st);
      const size_t cs = (size_t)Ms * d * es;  // candidate rows start here in A and Y
      if (r0 == 0) {
        hipError_t e = launch_gemm(bf, A, d, L.o.w, L.o.b, Xs, d, Ys[0], d, (int)Ms, d, d, EPI_BIAS_RESID, st);
        if (e != hipSuccess) return e;
      }
      return launch_gemm(bf, A + cs, d, L.o.w, L.o.b, Xc, d, Ys[0] + cs, d, (int)Mc, d, d, EPI_BIAS_RESID, st);
    }());
    TX_LAUNCH(K_LAYERNORM, 0, (fold ? 1 : 2) * Mrd * dd * esd,
              launch_layernorm(bf, Yk(k0), fold ? nullptr : T + ro, Sk(k0), L.ln1g, L.ln1b, Mr, d, eps, st));
    TX_LAUNCH(K_GEMM_XQ, xq.first, xq.second,
              fold ? launch_gemm(bf, Yk(k0), d, L.xqf.w, L.xqf.b, nullptr, 0, A + ro, d, Mr, d, d, EPI_LN, st,
                                 LnResid{Sk(k0), L.xqf.cs, nullptr})
                   : launch_gemm(bf, T + ro, d, L.xq.w, L.xq.b, nullptr, 0, A + ro, d, Mr, d, d, EPI_BIAS, st));
    TX_LAUNCH(K_CROSS_ATTN, 4 * dd * (last ? pairs_cand : pairs_full), kvb + 2 * Mrd * dd * esd,
              sparse ? launch_lg_attention(bf, A, d, O, d, c->pool, c->d_table, c->max_pages, c->geom, m->n_enc + l,
                                           areq, at, n_at, qb, m->l_local, m->gpool ? c->d_gkv : nullptr,
                                           2 * m->n_dec * d, l, st)
              : xpipe ? launch_cross_attention(
                            A, d, O, d, c->pool, c->d_table, c->max_pages, c->geom, m->n_enc + l,
                            (const XTile*)(ws + xd.wt), (const int32_t*)(ws + xd.wo), xp.whole.longest(),
                            (const XTile*)(ws + xd.st), (const int32_t*)(ws + xd.so), xp.split.longest(), xpart,
                            (const XMerge*)(ws + xd.mg), (int)xp.merges.size(), st)
                     : launch_paged_attention(bf, A, d, O, d, c->pool, c->d_table, c->max_pages, c->geom,
                                              m->n_enc + l, areq, at, n_at, false, nullptr, 0, qb, st));
    TX_LAUNCH(K_GEMM_XO, xo.first, xo.second,
              launch_gemm(bf, O + ro, d, L.xo.w, L.xo.b, Yk(k0), d, Yk(k0 + 1), d, Mr, d, d, EPI_BIAS_RESLN, st,
                          LnResid{Sk(k0), L.ln1g, L.ln1b}));
    TX_LAUNCH(K_LAYERNORM, 0, (fold ? 1 : 2) * Mrd * dd * esd,
              launch_layernorm(bf, Yk(k0 + 1), fold ? nullptr : T + ro, Sk(k0 + 1), L.ln2g, L.ln2b, Mr, d, eps, st));
    TX_LAUNCH(K_GEMM_FFN1, f1.first, f1.second,
              fold ? launch_gemm(bf, Yk(k0 + 1), d, L.f1f.w, L.f1f.b, nullptr, 0, Hf + (size_t)r0 * F * es, F, Mr, F,
                                 d, EPI_LN_GELU, st, LnResid{Sk(k0 + 1), L.f1f.cs, nullptr})
                   : launch_gemm(bf, T + ro, d, L.f1.w, L.f1.b, nullptr, 0, Hf + (size_t)r0 * F * es, F, Mr, F, d,
                                 EPI_BIAS_GELU, st));
    TX_LAUNCH(K_GEMM_FFN2, f2.first, f2.second,
              launch_gemm(bf, Hf + (size_t)r0 * F * es, F, L.f2.w, L.f2.b, Yk(k0 + 1), d, Yk(k0 + 2), d, Mr, d, F,
                          EPI_BIAS_RESLN, st, LnResid{Sk(k0 + 1), L.ln2g, L.ln2b}));
    if (last) {
      const int k = std::max(1, m->n_act);
      TX_LAUNCH(K_LN_SCORE, 2 * Mrd * dd * k, Mrd * dd * esd + 4 * Mrd * k,
                launch_layernorm_score(bf, Yk(k0 + 2), L.ln3g, L.ln3b, m->ws, m->bs, scores + (size_t)co[a] * k, Mr,
                                       d, eps, m->n_act, st));
    }
    else
      TX_LAUNCH(K_LAYERNORM, 0, (fold_out ? 1 : 2) * Mrd * dd * esd,
                launch_layernorm(bf, Yk(k0 + 2), fold_out ? nullptr : T + ro, Sk(k0 + 2), L.ln3g, L.ln3b, Mr, d,
                                 eps, st));
  }
  return TX_OK;
}

// Shared by score_candidates and score_events once ids and key lengths are
// checked: offsets, pointers, workspace, then the passes.
int score_groups(const tx_kv_cache* c, int n, const int32_t* ids, const int64_t* kvlen, const void* serving,
                 const int64_t* so, const void* cand, const int64_t* co, float* scores, void* ws, size_t ws_bytes,
                 hipStream_t st, bool fixed_staging = false) {
  TX_CHECK(check_offsets(so, n, "serving", 0));
  TX_CHECK(check_offsets(co, n, "candidate", 0));
  TX_CHECK(check_tokens(c, n, serving, so, "serving"));
  TX_CHECK(check_tokens(c, n, cand, co, "candidate"));
  if (co[n] > co[0] && !scores) return fail(TX_E_INVALID, "scores pointer is null");
  if (((uintptr_t)scores & 3)) return fail(TX_E_INVALID, "scores pointer misaligned");
  std::vector<int> cuts;
  TX_CHECK(plan_passes(c->m, TX_OP_SCORE, n, so, co, ws_bytes, cuts, fixed_staging ? kStagingReserve : SIZE_MAX));
  if (!ws) return fail(TX_E_INVALID, "workspace is null");
  TX_CHECK(check_weights(c));
  for (size_t p = 0; p + 1 < cuts.size(); ++p)
    TX_CHECK(run_score_pass(c, ids, kvlen, cuts[p], cuts[p + 1], (const char*)serving, so, (const char*)cand, co,
                            scores, (char*)ws, st, fixed_staging));
  return TX_OK;
}

}  // namespace

extern "C" {

int score_candidates(const tx_kv_cache* c, int32_t n, const int32_t* ids, const void* serving, const int64_t* so,
                     const void* cand, const int64_t* co, float* scores, void* ws, size_t ws_bytes, hipStream_t st) {
  TX_CHECK(common_checks(c, n, ids, ws));
  if (n == 0) return TX_OK;
  std::vector<int64_t> kvlen(n);
  for (int i = 0; i < n; ++i) {
    if (c->len[ids[i]] < 1) return fail(TX_E_NOCACHE, "request %d has no cache", ids[i]);
    kvlen[i] = c->len[ids[i]];
  }
  return score_groups(c, n, ids, kvlen.data(), serving, so, cand, co, scores, ws, ws_bytes, st);
}

int score_events(const tx_kv_cache* c, int32_t n, const int32_t* ids, const int64_t* prefix, const void* serving,
                 const int64_t* so, const void* cand, const int64_t* co, float* scores, void* ws, size_t ws_bytes,
                 hipStream_t st) {
  if (!c) return fail(TX_E_INVALID, "cache is null");
  if (n < 0) return fail(TX_E_INVALID, "n_events %d", n);
  if (n == 0) return TX_OK;
  if (!ids || !prefix) return fail(TX_E_INVALID, "event ids or prefix lengths are null");
  if (((uintptr_t)ws & 255)) return fail(TX_E_INVALID, "workspace not 256-byte aligned");
  for (int i = 0; i < n; ++i) {
    if (ids[i] < 0 || ids[i] >= c->max_req) return fail(TX_E_INVALID, "request id %d out of range", ids[i]);
    if (c->len[ids[i]] < 1) return fail(TX_E_NOCACHE, "request %d has no cache", ids[i]);
    if (prefix[i] < 1 || prefix[i] > c->len[ids[i]])
      return fail(TX_E_INVALID, "event %d: prefix %lld outside 1 .. %lld", i, (long long)prefix[i],
                  (long long)c->len[ids[i]]);
    if (c->m->gpool && prefix[i] != c->len[ids[i]])
      return fail(TX_E_UNSUPPORTED, "event %d: the pooled global token is kept for the whole cached history only",
                  i);
  }
  return score_groups(c, n, ids, prefix, serving, so, cand, co, scores, ws, ws_bytes, st);
}

int score_candidates_static(const tx_kv_cache* c, int32_t n, const int32_t* ids, const void* serving,
                            const int64_t* so, const void* cand, const int64_t* co, float* scores, hipStream_t st) {
  TX_CHECK(common_checks(c, n, ids, nullptr));
  if (n == 0) return TX_OK;
  std::vector<int64_t> kvlen(n);
  for (int i = 0; i < n; ++i) {
    if (c->len[ids[i]] < 1) return fail(TX_E_NOCACHE, "request %d has no cache", ids[i]);
    kvlen[i] = c->len[ids[i]];
  }
  if (!c->staging_reserved)
    return fail(TX_E_NOMEM, "no pinned staging was reserved when the cache was created (no usable device then)");
  int dev = -1;
  TX_HIP(hipGetDevice(&dev));
  if (st) {
    hipDevice_t sdev = -1;
    TX_HIP(hipStreamGetDevice(st, &sdev));
    if (sdev != dev) return fail(TX_E_INVALID, "stream belongs to device %d, the current device is %d", sdev, dev);
  }
  void* ws = nullptr;
  TX_HIP(static_scratch(&ws));
  return score_groups(c, n, ids, kvlen.data(), serving, so, cand, co, scores, ws, kStaticScratchBytes, st, true);
}

}  // extern "C"
