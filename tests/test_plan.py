"""Host checks of the attention work planner (paper_2605_31598_amd/csrc/plan.cpp).

The planner decides which query rows of which (layer, KV head) each attention
workgroup covers; a mistake there would make the kernel skip or repeat rows.
It is plain C++, so it is compiled here with g++ and run on the CPU:

* every query row of every (layer, KV head) is covered exactly once, by whole
  32-row waves, at most 8 waves per workgroup;
* row-tile slots of one (layer, KV head) are 0 .. tiles-1, each used once, and
  never more than plan_max_tiles (the size of the column-sum buffer);
* all work of one (layer, KV head) lands on one XCD (workgroup i runs on XCD i % 8);
* on each XCD the full workgroups come before the short ones;
* for the 7B-shaped 28-layer stack on 256 compute units the full workgroups fill
  exactly two rounds and the rest fits one round of short workgroups (at most
  four 32-row blocks), which are key-split when the caller allows it and never
  otherwise.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_31598_amd", "csrc")

DRIVER = r'''
#include <cstdio>
#include <cstdlib>
#include "plan.h"
int main(int argc, char** argv) {
  const int n_lg = atoi(argv[1]), rows = atoi(argv[2]), n_xcd = atoi(argv[3]), cu = atoi(argv[4]);
  const bool split_short = atoi(argv[5]) != 0;
  const int max_ks = atoi(argv[6]);
  const skv::AttnPlan p = skv::plan_attention(n_lg, rows, 32, 8, n_xcd, cu, split_short, max_ks);
  printf("bound %d\n", skv::plan_max_tiles(rows, 32, 8));
  printf("n_ks %d\n", p.n_ks);
  for (size_t i = 0; i < p.tiles.size(); ++i) printf("tiles %zu %d\n", i, p.tiles[i]);
  for (const auto& w : p.items) printf("item %d %d %d %d %d %d\n", w.lg, w.row0, w.rows, w.tile, w.split, w.ks);
  return 0;
}
'''


@pytest.fixture(scope="module")
def planner(tmp_path_factory):
    d = tmp_path_factory.mktemp("plan")
    src = d / "driver.cpp"
    src.write_text(DRIVER)
    exe = d / "driver"
    subprocess.run(["g++", "-O1", "-std=c++17", "-I", CSRC, str(src), os.path.join(CSRC, "plan.cpp"), "-o", str(exe)],
                   check=True)

    def run(n_lg, rows, n_xcd=8, cu_per_xcd=32, split_short=True, max_ks=1, with_ks=False):
        out = subprocess.run([str(exe), str(n_lg), str(rows), str(n_xcd), str(cu_per_xcd), str(int(split_short)),
                              str(max_ks)], capture_output=True, text=True, check=True).stdout.split("\n")
        bound = int(out[0].split()[1])
        n_ks = int(out[1].split()[1])
        tiles = [int(l.split()[2]) for l in out if l.startswith("tiles")]
        items = [tuple(int(x) for x in l.split()[1:]) for l in out if l.startswith("item")]
        if with_ks:
            return bound, n_ks, tiles, items
        assert n_ks == 1 and all(it[5] == 0 for it in items)
        return bound, tiles, [it[:5] for it in items]

    return run


SHAPES = [(112, 1372), (4, 1372), (640, 2048), (8, 2916), (2, 32), (28, 1372), (4, 196), (1, 37), (3, 1),
          (7, 7 * 196), (80, 2048 + 5), (13, 300), (9, 8 * 32 * 3 + 1)]


@pytest.mark.parametrize("n_lg,rows", SHAPES)
@pytest.mark.parametrize("n_xcd,cu", [(8, 32), (1, 4), (8, 1)])
@pytest.mark.parametrize("split_short", [True, False])
def test_plan_covers_every_row_once(planner, n_lg, rows, n_xcd, cu, split_short):
    bound, tiles, items = planner(n_lg, rows, n_xcd, cu, split_short)
    assert len(tiles) == n_lg
    covered = [[] for _ in range(n_lg)]
    slots = [set() for _ in range(n_lg)]
    xcd_of = {}
    for i, (lg, row0, nrows, tile, split) in enumerate(items):
        if nrows == 0:
            continue
        assert 0 <= lg < n_lg
        assert row0 % 32 == 0 and 0 < nrows <= 8 * 32 and row0 + nrows <= rows
        assert split in (0, 1) and (split == 0 or (split_short and nrows <= 4 * 32))
        assert nrows % 32 == 0 or row0 + nrows == rows  # only the last wave of a range is ragged
        covered[lg].append((row0, row0 + nrows))
        assert tile not in slots[lg]
        slots[lg].add(tile)
        assert xcd_of.setdefault(lg, i % n_xcd) == i % n_xcd, "one (layer, KV head) split over XCDs"
    for lg in range(n_lg):
        spans = sorted(covered[lg])
        assert spans[0][0] == 0 and spans[-1][1] == rows
        assert all(a[1] == b[0] for a, b in zip(spans, spans[1:])), f"gap or overlap in range {lg}"
        assert slots[lg] == set(range(tiles[lg]))
        assert tiles[lg] <= bound


@pytest.mark.parametrize("n_lg,rows", SHAPES)
def test_full_workgroups_first_on_each_xcd(planner, n_lg, rows):
    _, _, items = planner(n_lg, rows)
    for x in range(8):
        seq = [it for it in items[x::8] if it[2] > 0]
        full = [it[2] == 256 for it in seq]
        assert full == sorted(full, reverse=True)


@pytest.mark.parametrize("split_short", [True, False])
def test_7b_stack_two_full_rounds_then_short_round(planner, split_short):
    _, tiles, items = planner(28 * 4, 7 * 196, split_short=split_short)
    real = [it for it in items if it[2] > 0]
    full = [it for it in real if it[2] == 256]
    short = [it for it in real if it[2] < 256]
    assert len(full) == 2 * 256
    assert len(short) <= 256 and all(it[2] <= 4 * 32 for it in short)
    assert all(it[4] == 0 for it in full)
    assert all(it[4] == int(split_short) for it in short)
    assert max(tiles) <= 7


def test_small_call_uses_short_workgroups(planner):
    # one layer of the 7B shape: 43 wave blocks per KV head fit one round of short workgroups
    _, tiles, items = planner(4, 7 * 196)
    real = [it for it in items if it[2] > 0]
    assert all(it[2] <= 128 and it[4] == 1 for it in real)
    assert tiles == [11] * 4


# ---- key-split plans (calls too small to fill the device) ----

@pytest.mark.parametrize("n_lg,rows", [(4, 1372), (8, 1372), (12, 1372), (8, 2048), (1, 37), (3, 1), (2, 32 * 8 * 3)])
@pytest.mark.parametrize("n_xcd,cu", [(8, 32), (1, 4), (2, 8)])
@pytest.mark.parametrize("split_short", [True, False])
def test_key_split_plan_covers_rows_once_per_key_range(planner, n_lg, rows, n_xcd, cu, split_short):
    bound, n_ks, tiles, items = planner(n_lg, rows, n_xcd, cu, split_short, 16, with_ks=True)
    row_wgs = n_lg * -(-(-(-rows // 32)) // 8)  # full workgroups
    if 3 * row_wgs > n_xcd * cu:
        assert n_ks == 1
        return
    assert n_ks == min(16, n_xcd * cu // row_wgs) and n_ks >= 3
    covered = {}
    xcd_of = {}
    for i, (lg, row0, nrows, tile, split, ks) in enumerate(items):
        if nrows == 0:
            continue
        assert split == 0 and 0 <= ks < n_ks and 0 < nrows <= 256 and row0 % 32 == 0
        covered.setdefault((lg, ks), []).append((row0, row0 + nrows, tile))
        assert xcd_of.setdefault((lg, ks), i % n_xcd) == i % n_xcd, "one key range split over XCDs"
    assert set(covered) == {(lg, ks) for lg in range(n_lg) for ks in range(n_ks)}
    for (lg, ks), spans in covered.items():
        spans.sort()
        assert spans[0][0] == 0 and spans[-1][1] == rows
        assert all(a[1] == b[0] for a, b in zip(spans, spans[1:]))
        # the row tile slot of a row range is the same for every key range
        assert [sp[2] for sp in spans] == list(range(len(spans))) == list(range(tiles[lg]))
        assert tiles[lg] <= bound


def test_key_splits_for_one_layer_of_the_7b_stack(planner):
    # 4 (layer, KV head) ranges of 43 wave blocks: 24 row workgroups, 10 key ranges, all 8 XCDs busy
    _, n_ks, tiles, items = planner(4, 7 * 196, 8, 32, True, 16, with_ks=True)
    assert n_ks == 10 and tiles == [6] * 4
    real = [it for it in items if it[2] > 0]
    assert len(real) == 240 and all(it[4] == 0 for it in real)
    assert {i % 8 for i, it in enumerate(items) if it[2] > 0} == set(range(8))
    # the whole 28-layer stack fills the device without splitting keys
    _, n_ks, _, _ = planner(28 * 4, 7 * 196, 8, 32, True, 16, with_ks=True)
    assert n_ks == 1


SWEEP = r'''
#include <cstdio>
#include <vector>
#include "plan.h"
// Sweeps many shapes through the planner under AddressSanitizer and
// UndefinedBehaviorSanitizer, checking that every query row of every
// (layer, KV head) is covered exactly once per key split and that tile slots
// stay under plan_max_tiles.
int main() {
  const int rows_list[] = {1, 5, 31, 32, 33, 196, 255, 256, 257, 1372, 2048, 2916, 5000};
  long checked = 0;
  for (int n_lg : {1, 2, 3, 4, 7, 8, 16, 28, 112, 640})
    for (int rows : rows_list)
      for (int n_xcd : {1, 8})
        for (int cu : {1, 4, 32})
          for (int split_short : {0, 1})
            for (int max_ks : {1, 16}) {
              const skv::AttnPlan p = skv::plan_attention(n_lg, rows, 32, 8, n_xcd, cu, split_short != 0, max_ks);
              const int bound = skv::plan_max_tiles(rows, 32, 8);
              std::vector<int> cover(static_cast<size_t>(n_lg) * rows * p.n_ks, 0);
              for (const auto& w : p.items) {
                if (w.rows <= 0) continue;
                if (w.lg < 0 || w.lg >= n_lg || w.row0 < 0 || w.row0 + w.rows > rows || w.tile < 0 ||
                    w.tile >= bound || w.ks < 0 || w.ks >= p.n_ks) {
                  printf("bad item lg=%d row0=%d rows=%d tile=%d ks=%d\n", w.lg, w.row0, w.rows, w.tile, w.ks);
                  return 1;
                }
                for (int r = w.row0; r < w.row0 + w.rows; ++r)
                  ++cover[(static_cast<size_t>(w.lg) * p.n_ks + w.ks) * rows + r];
              }
              for (int c : cover)
                if (c != 1) {
                  printf("row covered %d times (n_lg=%d rows=%d)\n", c, n_lg, rows);
                  return 1;
                }
              if (static_cast<int>(p.tiles.size()) != n_lg) return 1;
              for (int t : p.tiles)
                if (t < 1 || t > bound) return 1;
              ++checked;
            }
  printf("checked %ld plans\n", checked);
  return 0;
}
'''


def test_planner_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    """The planner built with -fsanitize=address,undefined (host code only) over a sweep
    of shapes: no out-of-bounds access, overflow or other undefined behaviour, and every
    row covered once per key split."""
    src = tmp_path / "sweep.cpp"
    src.write_text(SWEEP)
    exe = tmp_path / "sweep"
    subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer", "-I", CSRC, str(src), os.path.join(CSRC, "plan.cpp"), "-o", str(exe)],
                   check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"})
    assert r.returncode == 0, r.stdout + r.stderr
    assert "checked" in r.stdout
