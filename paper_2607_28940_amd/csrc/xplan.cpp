// Host-side worklist of the pipelined decoder cross-attention (the work list
// of the scoring pass: (request, head, query block, kv-split) tiles).
#include <algorithm>
#include <cstdint>
#include <vector>

#include "tx_internal.h"
#include "xplan.h"

namespace tx {

// Worklist of the pipelined cross-attention (a1 of the scoring pass). Units
// are (request, head, 128-query block) against all the request's pages. When
// the batch leaves the GPU's resident blocks short of work, long units are
// split by pages (kv-split): a unit of P pages takes ceil(P / Q) parts of at
// least kXMinSplitPages, Q = the per-block share of all pages when every
// resident block has about two units; the parts' partial results are merged
// afterwards. Columns (request, head, part) group the query blocks that read
// the same pages; columns go to XCDs longest first (each XCD's least loaded
// first), and each XCD's list keeps a column's tiles adjacent, so that the
// resident blocks of one XCD read a page slab from its L2 close in time.
// Whole-request and kv-split columns form two tile sets, balanced apart.
void xattn_plan(const std::vector<AttnReq>& reqs, int H, int resident_blocks, int max_parts, XPlan& out) {
  struct Unit {
    int req, head, q0, qn, pages;
  };
  std::vector<Unit> units;
  int64_t work = 0;
  for (int r = 0; r < (int)reqs.size(); ++r) {
    const int nq = reqs[r].qa_n + reqs[r].qb_n;
    const int pages = (reqs[r].kv_len + kPage - 1) / kPage;
    if (nq <= 0 || pages <= 0) continue;
    for (int h = 0; h < H; ++h)
      for (int q0 = 0; q0 < nq; q0 += kXQueryBlock) {
        units.push_back({r, h, q0, std::min(kXQueryBlock, nq - q0), pages});
        work += pages;
      }
  }
  // page quantum: raised until the partial slots suffice
  int64_t quantum = std::max<int64_t>(kXMinSplitPages, (work + 2 * resident_blocks - 1) / (2 * resident_blocks));
  auto parts_of = [&](int pages) -> int {
    if (pages <= quantum) return 1;
    return (int)std::max<int64_t>(1, std::min<int64_t>((pages + quantum - 1) / quantum, pages / kXMinSplitPages));
  };
  for (;;) {
    int64_t n = 0;
    for (const Unit& u : units) {
      const int k = parts_of(u.pages);
      if (k > 1) n += k;
    }
    if (n <= max_parts) break;
    quantum *= 2;
  }
  // columns: (request, head, part) with their query blocks
  struct Column {
    int64_t cost;
    int first, count;  // units[first .. first + count) share request and head
    int part, n_parts, p0, p1;
  };
  std::vector<Column> cols;
  std::vector<int> unit_part0(units.size(), -1);
  int next_part = 0;
  for (int i = 0; i < (int)units.size();) {
    int j = i;
    while (j < (int)units.size() && units[j].req == units[i].req && units[j].head == units[i].head) ++j;
    const int pages = units[i].pages, k = parts_of(pages);
    for (int u = i; u < j; ++u) {
      if (k > 1) {
        unit_part0[u] = next_part;
        next_part += k;
      }
    }
    for (int part = 0; part < k; ++part) {
      const int p0 = (int)((int64_t)pages * part / k), p1 = (int)((int64_t)pages * (part + 1) / k);
      int64_t cost = 0;
      for (int u = i; u < j; ++u) cost += (int64_t)(p1 - p0) * 4 + 8;
      cols.push_back({cost, i, j - i, part, k, p0, p1});
    }
    i = j;
  }
  out.n_parts = next_part;
  std::stable_sort(cols.begin(), cols.end(), [](const Column& a, const Column& b) { return a.cost > b.cost; });
  std::vector<XTile> lists[2][8];
  int64_t load[2][8] = {};
  for (const Column& c : cols) {
    const int kind = c.n_parts > 1;
    int x = 0;
    for (int k = 1; k < 8; ++k)
      if (load[kind][k] < load[kind][x]) x = k;
    load[kind][x] += c.cost;
    for (int u = c.first; u < c.first + c.count; ++u) {
      const Unit& un = units[u];
      const AttnReq& rq = reqs[un.req];
      XTile t{};
      t.head = un.head;
      t.q_begin = un.q0;
      t.q_count = un.qn;
      t.part = kind ? unit_part0[u] + c.part : -1;
      t.page_begin = c.p0;
      t.page_end = c.p1;
      t.kv_len = rq.kv_len;
      t.slot = rq.slot;
      t.qa_row = rq.qa_row;
      t.qa_n = rq.qa_n;
      t.qb_row = rq.qb_row;
      lists[kind][x].push_back(t);
    }
  }
  for (int kind = 0; kind < 2; ++kind) {
    XTileSet& set = kind ? out.split : out.whole;
    set.tiles.clear();
    set.xoff.assign(9, 0);
    for (int x = 0; x < 8; ++x) {
      set.xoff[x] = (int32_t)set.tiles.size();
      set.tiles.insert(set.tiles.end(), lists[kind][x].begin(), lists[kind][x].end());
    }
    set.xoff[8] = (int32_t)set.tiles.size();
  }
  out.merges.clear();
  for (int u = 0; u < (int)units.size(); ++u) {
    if (unit_part0[u] < 0) continue;
    const Unit& un = units[u];
    const AttnReq& rq = reqs[un.req];
    out.merges.push_back({un.head, un.q0, un.qn, unit_part0[u], parts_of(un.pages), rq.qa_row, rq.qa_n, rq.qb_row});
  }
}

}  // namespace tx
