// Host-logic driver of the C ABI, run on a machine without a GPU against the
// real api.cpp linked with stub_kernels.cpp (launchers that do nothing), built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_harness.py. Covers argument checks, page bookkeeping, pass
// planning over many ragged requests and the failure path of a build or
// append whose first HIP call fails after the pages were assigned (here:
// the page-table upload, for want of a device).
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "transx.h"

static int g_fail = 0;
#define EXPECT(cond)                                                          \
  do {                                                                        \
    if (!(cond)) {                                                            \
      std::fprintf(stderr, "%s:%d: expected %s (last error: %s)\n", __FILE__, \
                   __LINE__, #cond, tx_last_error());                         \
      ++g_fail;                                                               \
    }                                                                         \
  } while (0)

// addresses that are never dereferenced on the host (the stubs launch nothing)
static void* fake(uintptr_t a) { return reinterpret_cast<void*>(a); }

static tx_config headline() {
  tx_config c{};
  c.d_model = 1024, c.n_heads = 8, c.d_ffn = 4096, c.n_enc_layers = 2, c.n_dec_layers = 2;
  c.rel_pos_buckets = 128, c.ln_eps = 1e-5f, c.dtype = TX_BF16;
  return c;
}

static int64_t len_of(tx_kv_cache* c, int id) {
  int64_t v = -7;
  EXPECT(tx_kv_cache_length(c, id, &v) == TX_OK);
  return v;
}

int main() {
  tx_config cfg = headline();
  const size_t rb = tx_model_repack_bytes(&cfg);
  EXPECT(rb > 0);
  tx_model* m = nullptr;
  EXPECT(tx_model_create(&cfg, fake(0x7E0000000000), rb, 7, &m) == TX_OK);
  // weights: the stub launchers accept any pointers
  const int nw = tx_num_weights(&cfg);
  std::vector<const void*> w(nw, fake(0x7F0000000000));
  EXPECT(tx_model_set_weights(m, w.data(), nw, nullptr) == TX_OK);

  const int64_t n_pages = 200;
  const int max_req = 64;
  const int64_t max_tokens = 3000;
  const size_t pb = tx_kv_pool_bytes(&cfg, n_pages, max_req, max_tokens);
  tx_kv_cache* c = nullptr;
  EXPECT(tx_kv_cache_create(m, fake(0x7D0000000000), pb, n_pages, max_req, max_tokens, &c) == TX_OK);
  EXPECT(tx_kv_cache_free_pages(c) == n_pages);

  void* X = fake(0x7C0000000000);
  void* ws = fake(0x7B0000000000);
  // argument errors change nothing
  {
    int32_t ids[2] = {3, 3};
    int64_t off[3] = {0, 10, 20};
    EXPECT(kv_cache_build(c, 2, ids, X, off, ws, (size_t)1 << 40, nullptr) == TX_E_INVALID);
    int32_t big[1] = {4};
    int64_t offb[2] = {0, 100 * 64 * 4};
    EXPECT(kv_cache_build(c, 1, big, X, offb, ws, (size_t)1 << 40, nullptr) == TX_E_INVALID);  // > max_tokens
    EXPECT(tx_kv_cache_free_pages(c) == n_pages);
  }
  // a build whose page-table upload fails after the pages were assigned:
  // the requests are left without a cache and keep their pages until release
  {
    int32_t ids[2] = {1, 2};
    int64_t off[3] = {0, 100, 300};  // 2 + 4 pages
    const int rc = kv_cache_build(c, 2, ids, X, off, ws, (size_t)1 << 40, nullptr);
    EXPECT(rc == TX_E_HIP);
    EXPECT(len_of(c, 1) == -1 && len_of(c, 2) == -1);
    EXPECT(tx_kv_cache_free_pages(c) == n_pages - 6);
    EXPECT(len_of(c, 0) == -1);
    EXPECT(tx_kv_cache_release(c, 2, ids) == TX_OK);
    EXPECT(tx_kv_cache_free_pages(c) == n_pages);
  }
  // append and score on requests without a cache: cold start
  {
    int32_t ids[1] = {5};
    int64_t off[2] = {0, 4};
    EXPECT(kv_cache_append(c, 1, ids, X, off, ws, (size_t)1 << 40, nullptr) == TX_E_NOCACHE);
    int64_t so[2] = {0, 3}, co[2] = {0, 5};
    EXPECT(score_candidates(c, 1, ids, X, so, X, co, (float*)fake(0x7A0000000000), ws, (size_t)1 << 40, nullptr) ==
           TX_E_NOCACHE);
    EXPECT(score_candidates_static(c, 1, ids, X, so, X, co, (float*)fake(0x7A0000000000), nullptr) == TX_E_NOCACHE);
  }
  // pass planning over many ragged requests: a workspace that holds a single
  // request makes every pass hold one; the minimum is the largest request
  {
    const int n = 64;
    std::vector<int64_t> so(n + 1), co(n + 1);
    so[0] = co[0] = 0;
    for (int i = 0; i < n; ++i) {
      so[i + 1] = so[i] + (i * 7) % 65;
      co[i + 1] = co[i] + 32 + (i * 389) % 993;
    }
    const size_t full = tx_workspace_bytes(c, TX_OP_SCORE, n, so.data(), co.data());
    const size_t one = tx_workspace_min_bytes(c, TX_OP_SCORE, n, so.data(), co.data());
    EXPECT(one > 0 && one < full);
    std::vector<int32_t> ids(n);
    for (int i = 0; i < n; ++i) ids[i] = i;
    // no request has a cache: reported before any planning or launch
    EXPECT(score_candidates(c, n, ids.data(), X, so.data(), X, co.data(), (float*)fake(0x7A0000000000), ws, one,
                            nullptr) == TX_E_NOCACHE);
  }
  // pool exhaustion
  {
    int32_t ids[1] = {9};
    int64_t off[2] = {0, (n_pages + 1) * 64};
    tx_kv_cache* small = nullptr;
    const size_t pb2 = tx_kv_pool_bytes(&cfg, 8, 4, 64 * 64);
    EXPECT(tx_kv_cache_create(m, fake(0x7D0000000000), pb2, 8, 4, 64 * 64, &small) == TX_OK);
    int32_t id0[1] = {0};
    int64_t off0[2] = {0, 9 * 64};
    EXPECT(kv_cache_build(small, 1, id0, X, off0, ws, (size_t)1 << 40, nullptr) == TX_E_NOMEM);
    EXPECT(tx_kv_cache_free_pages(small) == 8);
    (void)ids;
    (void)off;
    tx_kv_cache_destroy(small);
  }
  tx_kv_cache_destroy(c);
  tx_model_destroy(m);
  if (g_fail) {
    std::fprintf(stderr, "%d check(s) failed\n", g_fail);
    return 1;
  }
  std::printf("host harness: all checks passed\n");
  return 0;
}
