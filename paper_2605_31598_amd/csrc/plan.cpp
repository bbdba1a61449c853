// Attention work planner (see plan.h).
#include "plan.h"

#include <algorithm>

namespace skv {

namespace {

int ceil_div(int a, int b) { return (a + b - 1) / b; }

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
    out.push_back({lg, row0, row1 - row0, tiles[lg]++, key_split ? 1 : 0});
    b += nb;
  }
}

}  // namespace

AttnPlan plan_attention(int n_lg, int rows, int rows_per_wave, int max_waves, int n_xcd, int cu_per_xcd,
                        bool split_short) {
  AttnPlan plan;
  plan.tiles.assign(static_cast<size_t>(std::max(n_lg, 0)), 0);
  if (n_lg <= 0 || rows <= 0) return plan;
  n_xcd = std::max(n_xcd, 1);
  cu_per_xcd = std::max(cu_per_xcd, 1);
  const int nb = ceil_div(rows, rows_per_wave);  // wave blocks per range
  const int half = std::max(1, max_waves / 2);

  std::vector<std::vector<AttnWork>> lists(static_cast<size_t>(n_xcd));
  for (int x = 0; x < n_xcd; ++x) {
    const int lo = static_cast<int>(static_cast<int64_t>(x) * n_lg / n_xcd);
    const int hi = static_cast<int>(static_cast<int64_t>(x + 1) * n_lg / n_xcd);
    const int n = hi - lo;
    if (n == 0) continue;
    std::vector<AttnWork>& out = lists[static_cast<size_t>(x)];

    if (static_cast<int64_t>(n) * ceil_div(nb, half) <= cu_per_xcd) {  // one round of short workgroups
      for (int lg = lo; lg < hi; ++lg) split(out, plan.tiles, lg, 0, nb, half, rows, rows_per_wave, split_short);
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
        split(out, plan.tiles, lo + i, w * max_waves, max_waves, max_waves, rows, rows_per_wave, false);
    for (int i = 0; i < n; ++i) {
      const int first = keep[static_cast<size_t>(i)] * max_waves;
      split(out, plan.tiles, lo + i, first, nb - first, demote > 0 ? half : max_waves, rows, rows_per_wave,
            demote > 0 && split_short);
    }
  }
  size_t longest = 0;
  for (const auto& l : lists) longest = std::max(longest, l.size());
  plan.items.assign(longest * static_cast<size_t>(n_xcd), AttnWork{0, 0, 0, 0, 0});
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
