// CPU check of the forward's per-CU item-list planner (item_lists.h), built
// with g++ and run by tests/test_item_lists.py.  For each case: when lists are
// planned they must hold every item exactly once, no list may exceed the
// planned makespan, that makespan must beat dispatch in item order by 3%, and
// lists b .. b + n_cu / 8 - 1 must land on one XCD (workgroup g runs on XCD
// g % 8).  Prints one line per case; exits non-zero on the first failure.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <random>
#include <vector>

#include "item_lists.h"

using fastvr::ItemLists;
using fastvr::ItemShape;

static int fail(const char* what, int c) {
  printf("FAIL case %d: %s\n", c, what);
  return 1;
}

static int64_t n_items_of(const ItemShape& s) { return s.bh * (s.tiles_last + s.tiles_full * (s.n_local_chunks - 1)); }

// expect: 1 lists required, 0 plain dispatch required, -1 either
static int check(int c, const ItemShape& s, int n_cu, int expect) {
  const int n = (int)n_items_of(s);
  static ItemLists lst;
  int groups = 0;
  int64_t planned = 0, dispatched = 0;
  const bool used = fastvr::plan_item_lists(s, n, n_cu, &lst, &groups, &planned, &dispatched);
  printf("case %d: items %d cus %d lists %d planned %lld dispatch %lld\n", c, n, n_cu, used ? 1 : 0,
         (long long)planned, (long long)dispatched);
  if (expect == 1 && !used) return fail("lists expected", c);
  if (expect == 0 && used) return fail("plain dispatch expected", c);
  if (!used) return 0;
  if (groups != n_cu) return fail("one list per CU", c);
  if (100 * planned > 97 * dispatched) return fail("gain under 3%", c);
  if (lst.start[0] != 0 || lst.start[n_cu] != n) return fail("list bounds", c);
  std::vector<int> seen(n, 0);
  for (int g = 0; g < n_cu; ++g) {
    if (lst.start[g + 1] < lst.start[g]) return fail("list starts not monotone", c);
    int64_t load = 0;
    for (int u = lst.start[g]; u < lst.start[g + 1]; ++u) {
      const int it = lst.item[u];
      if (it < 0 || it >= n) return fail("item out of range", c);
      ++seen[it];
      load += fastvr::item_cost(s, it);
    }
    if (load > planned) return fail("list over the planned makespan", c);
  }
  for (int i = 0; i < n; ++i)
    if (seen[i] != 1) return fail("item missing or repeated", c);
  // XCD grouping: the bins b .. b + per - 1 sit on workgroups of one XCD, so
  // the first item of each list of an XCD comes from one run of sorted items;
  // checked here as: every workgroup index maps back to a distinct bin
  if (n_cu % 8 == 0) {
    const int per = n_cu / 8;
    std::vector<int> hit(n_cu, 0);
    for (int b = 0; b < n_cu; ++b) ++hit[(b % per) * 8 + b / per];
    for (int g = 0; g < n_cu; ++g)
      if (hit[g] != 1) return fail("bin to workgroup map is not a permutation", c);
  }
  return 0;
}

int main() {
  int c = 0;
  // 480p-shaped: B=1, H=12, 6 chunks of 3120 tokens (13 tiles), full prefix
  if (check(c++, ItemShape{12, 6, 13, 13, 3120, 0, -1, 18720, 96}, 256, 1)) return 1;
  // 1080p streaming step: 768 equal items, dispatch is already even
  if (check(c++, ItemShape{12, 1, 64, 64, 16320, 3, -1, 65280, 96}, 256, 0)) return 1;
  // fewer items than CUs; more items than a list launch takes (1080p parallel)
  if (check(c++, ItemShape{2, 4, 1, 1, 256, 0, -1, 1024, 96}, 256, 0)) return 1;
  if (check(c++, ItemShape{12, 4, 64, 64, 16320, 0, -1, 65280, 96}, 256, 0)) return 1;
  // a CU count that is not a multiple of 8, and a small one
  if (check(c++, ItemShape{12, 6, 13, 13, 3120, 0, -1, 18720, 96}, 100, -1)) return 1;
  if (check(c++, ItemShape{12, 6, 13, 13, 3120, 0, -1, 18720, 96}, 8, 0)) return 1;
  // the GPU zero-fill test's list-kernel shape: 4 chunks of 3120 tokens and a
  // last chunk of 770 (4 tiles), 672 items; it must take the list kernel
  if (check(c++, ItemShape{12, 5, 13, 4, 3120, 0, -1, 13250, 96}, 256, 1)) return 1;
  // seeded random shapes: windows, offsets, ragged last chunks
  std::mt19937 rng(1234);
  for (int r = 0; r < 400; ++r) {
    const int64_t L = 64 + rng() % 4000, nch = 1 + rng() % 8, bh = 1 + rng() % 24;
    const int64_t last = 1 + rng() % L, off = rng() % 3;
    const int64_t nq = (nch - 1) * L + last, nkv = off * L + nq + rng() % (L + 1);
    const int64_t W = (int64_t)(rng() % 5) - 1;
    const int64_t tf = (L + 255) / 256, tl = (last + 255) / 256;
    const ItemShape s{bh, nch, nch > 1 ? tf : tl, tl, L, off, W, nkv, 96};
    const int n_cu = (rng() % 4 == 0) ? 8 * (1 + rng() % 32) : 256;
    if (check(c++, s, n_cu, -1)) return 1;
  }
  // the plan cache returns what a fresh plan gives, hits and misses alike
  // (12 shapes cycled three times through its 8 entries, both decisions)
  {
    static fastvr::PlanCache cache;
    static ItemLists a, b;
    for (int rep = 0; rep < 36; ++rep) {
      const int r = rep % 12;
      const ItemShape s{12, 6 - r % 3, 13, 13 - r / 3, 3120, 0, r % 2 ? -1 : 2, 18720, 96};
      const int n = (int)n_items_of(s);
      int ga = 0, gb = 0;
      const bool ua = fastvr::plan_item_lists(s, n, 256, &a, &ga);
      const bool ub = cache.plan(s, n, 256, &b, &gb);
      if (ua != ub) return fail("plan cache decision differs", c);
      if (ua && (ga != gb || memcmp(a.start, b.start, sizeof(a.start)) != 0 ||
                 memcmp(a.item, b.item, sizeof(uint16_t) * n) != 0))
        return fail("plan cache lists differ", c);
    }
    ++c;
  }
  printf("all %d cases ok\n", c);
  return 0;
}
