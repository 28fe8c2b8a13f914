// Per-CU item lists for the forward kernel (host code, plain C++).
//
// The forward runs one workgroup per work item (a 256-row query tile of one
// batch, head and query chunk), dispatched longest first: the hardware hands
// the next workgroup to the first CU that frees up, which is list scheduling
// in item order.  When the items are only a few per CU and their lengths
// differ (short causal prefixes of early chunks next to long ones of late
// chunks), that can leave CUs idle at the end.  The alternative launches one
// workgroup per CU, each running a fixed list of items.  The lists come from
// first-fit decreasing into one bin per CU at the smallest capacity it fills,
// and are used only when their makespan beats dispatch by at least 3%.
#pragma once

#include <stdint.h>

#include <algorithm>
#include <mutex>

namespace fastvr {

constexpr int kListGroups = 256;    // workgroups of a list launch: at most one per CU
constexpr int kListMaxItems = 1024;

// Passed by value as a kernel argument (2.5 KB): workgroup g runs items
// item[start[g]] .. item[start[g + 1] - 1] in that order.
struct ItemLists {
  uint16_t start[kListGroups + 1];
  uint16_t item[kListMaxItems];
};

// What the item cost depends on: the forward's work decomposition.
struct ItemShape {
  int64_t bh;              // B * H
  int64_t n_local_chunks;  // query chunks of the call
  int64_t tiles_full;      // query tiles of a full chunk
  int64_t tiles_last;      // query tiles of the last chunk
  int64_t chunk_len, q_chunk_offset, window, nkv;  // window -1: unbounded
  int64_t key_tile;        // keys per K/V tile of the kernel
};

// Local query chunk of item vi.  Items are ordered last chunk first (the
// kernel's decode of an item index follows the same order).
inline int64_t item_chunk(const ItemShape& s, int64_t vi) {
  const int64_t n_last = s.bh * s.tiles_last;
  return vi < n_last ? s.n_local_chunks - 1 : s.n_local_chunks - 2 - (vi - n_last) / (s.bh * s.tiles_full);
}

// Work of item vi in key tiles, plus a fixed cost for its prologue and epilogue.
inline int64_t item_cost(const ItemShape& s, int64_t vi) {
  const int64_t cg = s.q_chunk_offset + item_chunk(s, vi);
  const int64_t L = s.chunk_len;
  const int64_t lo = (s.window >= 0 && cg > s.window) ? (cg - s.window) * L : 0;
  const int64_t hi = (L < s.nkv - cg * L) ? (cg + 1) * L : s.nkv;
  constexpr int64_t kItemOverhead = 2;
  return (hi - lo + s.key_tile - 1) / s.key_tile + kItemOverhead;
}

// Minimum load over n bins (segment tree): the leftmost bin whose load is at
// most `room`, and adding work to a bin.
struct MinTree {
  int n = 0, size = 1;
  int64_t t[2 * kListGroups];
  void init(int bins) {
    n = bins;
    size = 1;
    while (size < n) size *= 2;
    for (int i = 0; i < 2 * size; ++i) t[i] = (i >= size && i - size < n) ? 0 : INT64_MAX;
    for (int i = size - 1; i >= 1; --i) t[i] = std::min(t[2 * i], t[2 * i + 1]);
  }
  int leftmost_at_most(int64_t room) const {
    if (t[1] > room) return -1;
    int i = 1;
    while (i < size) i = (t[2 * i] <= room) ? 2 * i : 2 * i + 1;
    return i - size;
  }
  void add(int bin, int64_t w) {
    int i = bin + size;
    t[i] += w;
    for (i /= 2; i >= 1; i /= 2) t[i] = std::min(t[2 * i], t[2 * i + 1]);
  }
};

// First fit of items with the given costs (longest first) into `bins` bins of
// capacity cap; bin_of[k] receives the bin of item k.
inline bool first_fit(const int64_t* cost, int n, int bins, int64_t cap, MinTree& tree, int16_t* bin_of) {
  tree.init(bins);
  for (int k = 0; k < n; ++k) {
    const int b = tree.leftmost_at_most(cap - cost[k]);
    if (b < 0) return false;
    tree.add(b, cost[k]);
    bin_of[k] = (int16_t)b;
  }
  return true;
}

// Plans the lists for n_items items on n_cu CUs.  Returns false (keep plain
// dispatch) when there are too few or too many items or the gain is under 3%.
// *planned and *dispatched receive the two makespans (in key tiles) when not
// null, whatever the decision.
inline bool plan_item_lists(const ItemShape& s, int n_items, int n_cu, ItemLists* out, int* n_groups,
                            int64_t* planned = nullptr, int64_t* dispatched = nullptr) {
  if (planned) *planned = 0;
  if (dispatched) *dispatched = 0;
  if (n_items <= n_cu || n_items > kListMaxItems || n_cu < 8 || n_cu > kListGroups) return false;
  int64_t cost[kListMaxItems];
  int64_t total = 0, longest = 0;
  for (int vi = 0; vi < n_items; ++vi) {
    cost[vi] = item_cost(s, vi);
    total += cost[vi];
    longest = std::max(longest, cost[vi]);
  }
  // dispatch in item order: each item starts on the CU that frees up first
  MinTree tree;
  tree.init(n_cu);
  int64_t dispatch = 0;
  for (int vi = 0; vi < n_items; ++vi) {
    const int64_t least = tree.t[1];
    tree.add(tree.leftmost_at_most(least), cost[vi]);
    dispatch = std::max(dispatch, least + cost[vi]);
  }
  if (dispatched) *dispatched = dispatch;
  // items by cost, longest first; equal costs keep item order, so neighbours
  // in a list share their K/V stream
  int16_t order[kListMaxItems];
  for (int k = 0; k < n_items; ++k) order[k] = (int16_t)k;
  std::stable_sort(order, order + n_items, [&](int16_t x, int16_t y) { return cost[x] > cost[y]; });
  int64_t sorted_cost[kListMaxItems];
  for (int k = 0; k < n_items; ++k) sorted_cost[k] = cost[order[k]];
  // the smallest capacity first fit fills, by bisection below the dispatch makespan
  int64_t lo = std::max((total + n_cu - 1) / n_cu, longest), hi = dispatch;
  int16_t bin_of[kListMaxItems], best[kListMaxItems];
  bool found = false;
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (first_fit(sorted_cost, n_items, n_cu, mid, tree, bin_of)) {
      found = true;
      hi = mid;
      std::copy(bin_of, bin_of + n_items, best);
    } else {
      lo = mid + 1;
    }
  }
  if (!found) return false;
  if (planned) *planned = hi;
  if (100 * hi > 97 * dispatch) return false;
  // Workgroups go to the 8 XCDs round-robin: bin b runs as workgroup
  // (b % per) * 8 + b / per, so bins b .. b + per - 1 share an XCD and its L2.
  const int per = n_cu % 8 == 0 ? n_cu / 8 : n_cu;
  int count[kListGroups] = {};
  for (int k = 0; k < n_items; ++k) ++count[best[k]];
  int bin_at_wg[kListGroups], fill[kListGroups];
  for (int b = 0; b < n_cu; ++b) bin_at_wg[per == n_cu ? b : (b % per) * 8 + b / per] = b;
  out->start[0] = 0;
  for (int g = 0; g < n_cu; ++g) {
    out->start[g + 1] = (uint16_t)(out->start[g] + count[bin_at_wg[g]]);
    fill[bin_at_wg[g]] = out->start[g];
  }
  for (int k = 0; k < n_items; ++k) out->item[fill[best[k]]++] = (uint16_t)order[k];
  *n_groups = n_cu;
  return true;
}

inline bool same_shape(const ItemShape& a, const ItemShape& b) {
  return a.bh == b.bh && a.n_local_chunks == b.n_local_chunks && a.tiles_full == b.tiles_full &&
         a.tiles_last == b.tiles_last && a.chunk_len == b.chunk_len && a.q_chunk_offset == b.q_chunk_offset &&
         a.window == b.window && a.nkv == b.nkv && a.key_tile == b.key_tile;
}

// The last few plans (positive and negative decisions alike), so that a caller
// repeating one call shape plans it once.  Thread-safe; entries are replaced
// round-robin.  A plan depends only on the shape, the item count and the CU
// count, all part of the key.
class PlanCache {
 public:
  static constexpr int kEntries = 8;
  bool plan(const ItemShape& s, int n_items, int n_cu, ItemLists* out, int* n_groups) {
    {
      std::lock_guard<std::mutex> g(mu_);
      for (int e = 0; e < kEntries; ++e) {
        const Entry& x = ent_[e];
        if (x.valid && x.n_items == n_items && x.n_cu == n_cu && same_shape(x.shape, s)) {
          if (x.used) {
            *out = x.lists;
            *n_groups = x.n_groups;
          }
          return x.used;
        }
      }
    }
    Entry fresh;
    fresh.shape = s;
    fresh.n_items = n_items;
    fresh.n_cu = n_cu;
    fresh.used = plan_item_lists(s, n_items, n_cu, &fresh.lists, &fresh.n_groups);
    fresh.valid = true;
    if (fresh.used) {
      *out = fresh.lists;
      *n_groups = fresh.n_groups;
    }
    std::lock_guard<std::mutex> g(mu_);
    ent_[next_] = fresh;
    next_ = (next_ + 1) % kEntries;
    return fresh.used;
  }

 private:
  struct Entry {
    ItemShape shape{};
    int n_items = 0, n_cu = 0, n_groups = 0;
    bool valid = false, used = false;
    ItemLists lists;
  };
  std::mutex mu_;
  Entry ent_[kEntries];
  int next_ = 0;
};

}  // namespace fastvr
