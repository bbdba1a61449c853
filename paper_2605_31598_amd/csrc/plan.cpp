// Attention work planner (see plan.h).
#include "plan.h"

#include <algorithm>

namespace skv {

namespace {

int ceil_div(int a, int b) { return (a + b - 1) / b; }

typedef std::vector<std::vector<AttnWork>> XcdLists;

// Appends ceil(blocks / max_chunk) workgroups of nearly equal block counts
// covering blocks [first, first + blocks) of range lg.
void split(std::vector<AttnWork>& out, std::vector<int32_t>& tiles, int lg, int first, int blocks, int max_chunk,
           int rows, int rpw, bool key_split) {
  if (blocks <= 0) return;
  const int n = ceil_div(blocks, max_chunk);
  int b = first;
  for (int i = 0; i < n; ++i) {
    const int nb = blocks / n + (i < blocks % n ? 1 : 0);
    const int row0 = b * rpw;
    const int row1 = std::min(rows, (b + nb) * rpw);
    out.push_back({lg, row0, row1 - row0, tiles[lg]++, key_split ? 1 : 0, 0});
    b += nb;
  }
}

// Small calls: every range cut into workgroups of `chunk` row blocks (with
// key_halves, half-size workgroups whose waves share rows), each repeated for
// n_ks key ranges; group (lg, ks) on XCD (lg * n_ks + ks) % n_xcd.
void plan_key_splits(AttnPlan& plan, XcdLists& lists, int n_lg, int rows, int rpw, int chunk, bool key_halves,
                     int n_ks) {
  const int n_xcd = static_cast<int>(lists.size());
  const int nb = ceil_div(rows, rpw);
  plan.n_ks = n_ks;
  for (int lg = 0; lg < n_lg; ++lg) {
    for (int ks = 0; ks < n_ks; ++ks) {
      std::vector<AttnWork>& out = lists[static_cast<size_t>((static_cast<int64_t>(lg) * n_ks + ks) % n_xcd)];
      int tile = 0;
      for (int b = 0; b < nb; b += chunk) {
        const int row0 = b * rpw;
        const int row1 = std::min(rows, (b + chunk) * rpw);
        out.push_back({lg, row0, row1 - row0, tile++, key_halves ? 1 : 0, ks});
      }
      plan.tiles[static_cast<size_t>(lg)] = tile;
    }
  }
}

// Whole key ranges: the ranges split evenly over the XCDs, full workgroups in
// whole rounds first, short ones (split when split_short) in the last round.
void plan_rounds(AttnPlan& plan, XcdLists& lists, int n_lg, int rows, int rpw, int max_waves, int cu_per_xcd,
                 bool split_short) {
  const int n_xcd = static_cast<int>(lists.size());
  const int nb = ceil_div(rows, rpw);
  const int half = std::max(1, max_waves / 2);
  for (int x = 0; x < n_xcd; ++x) {
    const int lo = static_cast<int>(static_cast<int64_t>(x) * n_lg / n_xcd);
    const int hi = static_cast<int>(static_cast<int64_t>(x + 1) * n_lg / n_xcd);
    const int n = hi - lo;
    if (n == 0) continue;
    std::vector<AttnWork>& out = lists[static_cast<size_t>(x)];

    if (static_cast<int64_t>(n) * ceil_div(nb, half) <= cu_per_xcd) {  // one round of short workgroups
      for (int lg = lo; lg < hi; ++lg) split(out, plan.tiles, lg, 0, nb, half, rows, rpw, split_short);
      continue;
    }
    const int q = nb / max_waves, r = nb % max_waves;
    const int64_t full = static_cast<int64_t>(n) * q;
    // full workgroups to break up so that the full ones fill whole rounds
    int64_t demote = 0;
    if (full > cu_per_xcd && full % cu_per_xcd != 0) {
      const int64_t d = full % cu_per_xcd;
      int64_t short_count = 0;
      bool ok = true;
      for (int i = 0; i < n; ++i) {
        const int64_t di = d / n + (i < d % n ? 1 : 0);
        if (di > q) ok = false;
        short_count += ceil_div(static_cast<int>(r + max_waves * di), half);
      }
      if (ok && short_count <= cu_per_xcd) demote = d;
    }
    std::vector<int> keep(static_cast<size_t>(n));
    for (int i = 0; i < n; ++i) {
      const int64_t di = demote / n + (i < demote % n ? 1 : 0);
      keep[static_cast<size_t>(i)] = q - static_cast<int>(di);
    }
    for (int i = 0; i < n; ++i)
      for (int w = 0; w < keep[static_cast<size_t>(i)]; ++w)
        split(out, plan.tiles, lo + i, w * max_waves, max_waves, max_waves, rows, rpw, false);
    for (int i = 0; i < n; ++i) {
      const int first = keep[static_cast<size_t>(i)] * max_waves;
      split(out, plan.tiles, lo + i, first, nb - first, demote > 0 ? half : max_waves, rows, rpw,
            demote > 0 && split_short);
    }
  }
}

}  // namespace

AttnPlan plan_attention(int n_lg, int rows, int rows_per_wave, int max_waves, int n_xcd, int cu_per_xcd,
                        bool split_short, int max_key_splits) {
  AttnPlan plan;
  plan.tiles.assign(static_cast<size_t>(std::max(n_lg, 0)), 0);
  if (n_lg <= 0 || rows <= 0) return plan;
  n_xcd = std::max(n_xcd, 1);
  cu_per_xcd = std::max(cu_per_xcd, 1);

  XcdLists lists(static_cast<size_t>(n_xcd));
  // key-split plans use full workgroups: a key range is a few tiles, and the
  // per-tile costs of a workgroup do not shrink with its rows
  const int64_t row_wgs = static_cast<int64_t>(n_lg) * ceil_div(ceil_div(rows, rows_per_wave), max_waves);
  const int64_t n_cu = static_cast<int64_t>(n_xcd) * cu_per_xcd;
  if (max_key_splits > 1 && 3 * row_wgs <= n_cu)
    plan_key_splits(plan, lists, n_lg, rows, rows_per_wave, max_waves, false,
                    static_cast<int>(std::min<int64_t>(max_key_splits, n_cu / row_wgs)));
  else
    plan_rounds(plan, lists, n_lg, rows, rows_per_wave, max_waves, cu_per_xcd, split_short);

  size_t longest = 0;
  for (const auto& l : lists) longest = std::max(longest, l.size());
  plan.items.assign(longest * static_cast<size_t>(n_xcd), AttnWork{0, 0, 0, 0, 0, 0});
  for (size_t j = 0; j < longest; ++j)
    for (int x = 0; x < n_xcd; ++x)
      if (j < lists[static_cast<size_t>(x)].size())
        plan.items[j * static_cast<size_t>(n_xcd) + static_cast<size_t>(x)] = lists[static_cast<size_t>(x)][j];
  return plan;
}

int plan_max_tiles(int rows, int rows_per_wave, int max_waves) {
  if (rows <= 0) return 0;
  return ceil_div(ceil_div(rows, rows_per_wave), std::max(1, max_waves / 2));
}

}  // namespace skv
