"""The benchmark's bookkeeping of sampled stage events (host logic, no GPU)."""
from __future__ import annotations

import bench


def _slots(n_streams, first, last):
    return [(i, f) for i in range(n_streams) for f in range(first, last)]


def test_stride_one_keeps_every_step():
    rec = _slots(2, 11, 20)
    got = bench.sampled_frames(rec, 1)
    assert got == {0: list(range(9)), 1: list(range(9, 18))}


def test_stride_counts_each_stream_from_its_first_step():
    # two streams of 501 state-full frames each, 2048 steps: the second stream
    # starts counting again at its own first step, as each context's stride does
    rec = _slots(5, 11, 512)[:2048]
    got = bench.sampled_frames(rec, 8)
    assert got[0] == list(range(0, 501, 8))
    assert got[1] == list(range(501, 1002, 8))
    assert got[4] == [g for g in range(2004, 2048) if (g - 2004) % 8 == 0]
    assert sum(len(v) for v in got.values()) == sum(-(-n // 8) for n in (501, 501, 501, 501, 44))


def test_rows_of_timed_frames_follow_stream_order():
    # rows of the concatenated event arrays are ordered stream by stream; the timed
    # ones are those whose step index is past the warm-up
    rec = _slots(5, 11, 512)[:2048]
    warmup, stride = 512, 8
    got = bench.sampled_frames(rec, stride)
    order = [g for i in sorted(got) for g in got[i]]
    timed = [g for g in order if g >= warmup]
    assert timed == sorted(timed) and all(g >= warmup for g in timed)
    assert len(timed) == len([g for g in range(warmup, 2048) if (g - 501 * (g // 501)) % stride == 0]) == 193
