// Host-logic driver of the C ABI, run on a machine without a GPU against the
// real api.cpp linked with stub_kernels.cpp (launchers that do nothing), built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_harness.py. Covers argument checks, page bookkeeping, pass
// planning over many ragged requests and the failure path of a build or
// append whose first HIP call fails after the pages were assigned (here:
// the page-table upload, for want of a device).
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "transx.h"
#include "../../paper_2607_28940_amd/csrc/xplan.h"

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


// Properties of the cross-attention work list for one set of requests.
// expect_split: 1 = some unit is split, 0 = none, -1 = either
static void check_plan(const std::vector<tx::AttnReq>& reqs, int H, int blocks, int max_parts, int expect_split) {
  tx::XPlan p;
  tx::xattn_plan(reqs, H, blocks, max_parts, p);
  EXPECT(p.n_parts <= max_parts);
  // coverage[r][h][q][page]: how often the pair is computed
  std::vector<std::vector<int>> cover(reqs.size() * H);
  std::vector<int> part_use(p.n_parts, 0);
  bool split = false;
  for (int kind = 0; kind < 2; ++kind) {
    const tx::XTileSet& set = kind ? p.split : p.whole;
    EXPECT(set.xoff.size() == 9 && set.xoff[0] == 0 && set.xoff[8] == (int)set.tiles.size());
    for (int x = 0; x < 8 && set.xoff.size() == 9; ++x) EXPECT(set.xoff[x] <= set.xoff[x + 1]);
    int longest = 0;
    for (int x = 0; x < 8 && set.xoff.size() == 9; ++x) longest = std::max(longest, set.xoff[x + 1] - set.xoff[x]);
    EXPECT(set.longest() == longest);
    for (const tx::XTile& t : set.tiles) {
      int r = -1;
      for (int i = 0; i < (int)reqs.size(); ++i)
        if (reqs[i].slot == t.slot) r = i;
      EXPECT(r >= 0);
      if (r < 0) continue;
      const tx::AttnReq& q = reqs[r];
      const int nq = q.qa_n + q.qb_n, pages = (q.kv_len + 63) / 64;
      EXPECT(t.head >= 0 && t.head < H && t.q_count >= 1 && t.q_count <= tx::kXQueryBlock);
      EXPECT(t.q_begin >= 0 && t.q_begin + t.q_count <= nq && t.q_begin % tx::kXQueryBlock == 0);
      EXPECT(t.page_begin >= 0 && t.page_begin < t.page_end && t.page_end <= pages);
      EXPECT(t.kv_len == q.kv_len && t.qa_row == q.qa_row && t.qa_n == q.qa_n && t.qb_row == q.qb_row);
      EXPECT((t.part >= 0) == (kind == 1));  // each kind in its own set
      if (t.part >= 0) {
        split = true;
        EXPECT(t.part < p.n_parts);
        if (t.part < p.n_parts) ++part_use[t.part];
        EXPECT(t.page_end - t.page_begin >= tx::kXMinSplitPages);
      } else {
        EXPECT(t.page_begin == 0 && t.page_end == pages);
      }
      std::vector<int>& cv = cover[(size_t)r * H + t.head];
      cv.resize((size_t)nq * pages, 0);
      for (int i = t.q_begin; i < t.q_begin + t.q_count; ++i)
        for (int pg = t.page_begin; pg < t.page_end; ++pg) ++cv[(size_t)i * pages + pg];
    }
  }
  if (expect_split >= 0) EXPECT(split == (expect_split == 1));
  for (int s = 0; s < p.n_parts; ++s) EXPECT(part_use[s] == 1);
  for (int r = 0; r < (int)reqs.size(); ++r) {
    const int nq = reqs[r].qa_n + reqs[r].qb_n, pages = (reqs[r].kv_len + 63) / 64;
    for (int h = 0; h < H; ++h) {
      const std::vector<int>& cv = cover[(size_t)r * H + h];
      EXPECT(cv.size() == (size_t)nq * pages);
      for (int v : cv) EXPECT(v == 1);
    }
  }
  // merges: one per split (request, head, query block), covering its part slots
  std::vector<int> merged(p.n_parts, 0);
  for (const tx::XMerge& mg : p.merges) {
    EXPECT(mg.n_parts >= 2 && mg.part0 >= 0 && mg.part0 + mg.n_parts <= p.n_parts);
    for (int k = 0; k < mg.n_parts && mg.part0 + k < p.n_parts; ++k) ++merged[mg.part0 + k];
  }
  for (int s = 0; s < p.n_parts; ++s) EXPECT(merged[s] == 1);
}

static void check_plans() {
  std::vector<tx::AttnReq> reqs;
  // headline-like batch: no request is split
  for (int r = 0; r < 64; ++r) reqs.push_back({r * 576, 64, 64 * 576 + r * 512, 512, 4096, 0, r, 0});
  check_plan(reqs, 8, 512, 512, 0);
  // four long requests with a ragged tail page: split, every part >= 16 pages
  reqs.clear();
  for (int r = 0; r < 4; ++r) reqs.push_back({r * 600, 64, 4 * 600 + r * 536, 536 + r, 16384 - 37 * r, 0, 10 + r, 0});
  check_plan(reqs, 8, 512, 512, 1);
  // the same with too few partial slots for any split: the quantum grows
  // past the longest unit
  check_plan(reqs, 8, 512, 40, 0);
  // one long request, two heads, one query block: 32 slots suffice
  reqs.assign(1, tx::AttnReq{0, 30, 30, 70, 16384, 0, 2, 0});
  check_plan(reqs, 2, 512, 40, 1);
  // one request, one head, one query, short cache: a single tile
  reqs.assign(1, tx::AttnReq{5, 1, 0, 0, 100, 0, 3, 0});
  check_plan(reqs, 1, 512, 512, 0);
  // ragged mix, no candidates for some requests
  reqs.clear();
  uint32_t z = 12345;
  auto rnd = [&](int n) { z = z * 1664525u + 1013904223u; return (int)((z >> 8) % (uint32_t)n); };
  int row = 0;
  for (int r = 0; r < 40; ++r) {
    const int S = rnd(65), C = rnd(300), L = 1 + rnd(9000);
    reqs.push_back({row, S, row + S, C, L, 0, r, 0});
    row += S + C;
  }
  check_plan(reqs, 4, 64, 512, -1);
}

int main() {
  check_plans();
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
