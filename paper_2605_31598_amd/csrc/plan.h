// Host-side work plan of the attention launch: which query rows of which
// (layer, KV head) each workgroup processes, in launch order.
//
// Plain C++ (no HIP types) so that the planner also builds and runs on a host
// without a GPU.
#pragma once

#include <stdint.h>

#include <vector>

namespace skv {

// One workgroup's share: rows [row0, row0 + rows) of the packed G*T query rows
// of (layer, KV head) `lg`; its column sums of P go to row-tile slot `tile`.
// rows == 0 marks an empty slot (the workgroup exits at once).  split != 0: at
// most half a workgroup of row blocks, each covered by two waves that take one
// half of every key tile each (two waves per SIMD on a short share of rows).
struct AttnWork {
  int32_t lg, row0, rows, tile, split;
  int32_t ks;  // key split: the workgroup covers key tiles [ks * n / n_ks, (ks + 1) * n / n_ks)
};

struct AttnPlan {
  std::vector<AttnWork> items;  // one per workgroup, in launch order
  std::vector<int32_t> tiles;   // row tiles written for each (layer, KV head)
  int32_t n_ks = 1;             // key splits (> 1: statistics, output and combine launches)
};

// Splits n_lg ranges of `rows` query rows into workgroups of at most
// `max_waves` waves of `rows_per_wave` rows.
//
// The device runs one workgroup per compute unit at a time and dispatches
// workgroup i to XCD i % n_xcd; each XCD has cu_per_xcd compute units and its
// own L2.  Every (layer, KV head) stays on one XCD (its K/V rows are fetched
// into that L2 once), and each XCD's list holds its full workgroups first and
// its partial ones last.  When the full workgroups do not fill whole rounds of
// the XCD's compute units, enough of them are broken into short workgroups of
// at most max_waves/2 row blocks that the last round holds only such short
// workgroups.  If every range fits into one round of short workgroups, all
// workgroups are short.  With split_short, short workgroups are marked split
// (two waves per row block, one per key half); otherwise they run one wave per
// row block.
//
// Calls too small to fill the device (full row workgroups for at most a third
// of its compute units, up to max_key_splits > 1) split the keys instead: each
// full row workgroup is repeated for n_ks key ranges, and the (layer-head, key
// range) groups go round-robin over the XCDs.
AttnPlan plan_attention(int n_lg, int rows, int rows_per_wave, int max_waves, int n_xcd, int cu_per_xcd,
                        bool split_short, int max_key_splits);

// Upper bound on plan.tiles[i] for any n_lg, n_xcd and cu_per_xcd.
int plan_max_tiles(int rows, int rows_per_wave, int max_waves);

}  // namespace skv
