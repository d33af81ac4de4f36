// Worklist of the pipelined decoder cross-attention, built on the host.
#pragma once

#include <cstdint>
#include <vector>

#include "tx_internal.h"

namespace tx {

// One tile set per kind: whole-request tiles (rows written normalised) and
// kv-split tiles (partial slots, merged afterwards); each is a per-XCD list
// set of its own, balanced on its own, for a launch of its own.
struct XTileSet {
  std::vector<XTile> tiles;   // per-XCD lists, concatenated
  std::vector<int32_t> xoff;  // 9 entries: XCD x owns tiles[xoff[x] .. xoff[x + 1])
  int longest() const {
    int n = 0;
    for (int x = 0; x + 1 < (int)xoff.size(); ++x) n = n > xoff[x + 1] - xoff[x] ? n : xoff[x + 1] - xoff[x];
    return n;
  }
};
struct XPlan {
  XTileSet whole, split;
  std::vector<XMerge> merges;
  int n_parts = 0;  // partial slots used (kv-split tiles)
};

// Fewest pages a kv-split part covers.
constexpr int kXMinSplitPages = 16;

// Tiles for the requests of one cross-attention launch (queries of request r:
// reqs[r].qa_n + reqs[r].qb_n, keys: its first kv_len cached tokens) on a GPU
// with `resident_blocks` resident blocks, using at most max_parts partial
// slots.
void xattn_plan(const std::vector<AttnReq>& reqs, int H, int resident_blocks, int max_parts, XPlan& out);

}  // namespace tx
