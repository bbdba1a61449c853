"""The three key-split schemes of small calls, through the C ABI.

A call too small to fill the device splits the attention's keys into ranges
whose row statistics are merged before the output is formed.  key_split_mode 0
does it in one launch whose workgroups exchange the statistics (waiting a
bounded time for each other and computing what has not arrived), 1 in two
launches, 2 in one launch in which every workgroup computes every range itself
(the exchange's fallback for every range).  All three must give the same
outputs, states, scores, candidate pools and decode-cache rows, bit for bit:
on a single-layer model (the 7B-shaped layer, one call per frame), on a 7B-shaped
stack stepped one layer per call (whose selections ride in the next call's
attention launch), and on a 72B-shaped stack stepped one layer per call, whose
key-split launch has as many workgroups as the device has compute units.
"""
from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2605_31598_amd import FrameStepper  # noqa: E402
from workloads import WorkloadConfig  # noqa: E402

from .gpu_harness import frame_tensors, say  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


def _run_modes(wl, per_layer, modes=(0, 1, 2)):
    L, Hq, T, d = wl.n_layers, wl.n_q_heads, wl.tokens_per_frame, wl.head_dim
    st = [FrameStepper.from_workload(wl, key_split_mode=m) for m in modes]
    try:
        outs = [torch.empty((L, Hq, T, d), dtype=torch.bfloat16, device="cuda") for _ in modes]
        for n in range(wl.n_frames):
            q, k, v, _ = frame_tensors(wl, n, list(range(L)))
            spans = [(l, 1) for l in range(L)] if per_layer else [(0, L)]
            for s, o in zip(st, outs):
                for l0, lc in spans:
                    sl = slice(l0, l0 + lc)
                    s.step(q[sl], k[sl], v[sl], o[sl], layer_begin=l0, layer_count=lc)
            torch.cuda.synchronize()
            for m, o in zip(modes[1:], outs[1:]):
                assert torch.equal(outs[0].view(torch.int16), o.view(torch.int16)), \
                    f"{wl.name} frame {n}: output of key_split_mode {m}"
            if n % 2 == 1 or n == wl.n_frames - 1:
                for l in range(L):
                    ref = st[0].read_state(l)
                    for m, s in zip(modes[1:], st[1:]):
                        got = s.read_state(l)
                        for key in ("pos", "score", "k", "v", "pool_score", "pool_pos"):
                            assert np.array_equal(ref[key], got[key]), \
                                f"{wl.name} frame {n}: {key} of layer {l}, key_split_mode {m}"
                    ca = st[0].read_cache(l)
                    for m, s in zip(modes[1:], st[1:]):
                        cb = s.read_cache(l)
                        assert ca[2] == cb[2] and np.array_equal(ca[0], cb[0]) and np.array_equal(ca[1], cb[1]), \
                            f"{wl.name} frame {n}: decode cache of layer {l}, key_split_mode {m}"
        say(f"{wl.name}: {wl.n_frames} frames equal under key_split_mode {modes}")
    finally:
        for s in st:
            s.close()


def test_key_split_modes_agree_single_layer_model():
    _run_modes(WorkloadConfig("ks_7b_layer", 1, 28, 4, 128, 196, 8, 1024, "bf16", "iid", 9200), False)


def test_key_split_modes_agree_7b_stack_one_layer_per_call():
    _run_modes(WorkloadConfig("ks_7b_stack", 3, 28, 4, 128, 196, 8, 1024, "bf16", "iid", 9201), True)


def test_key_split_modes_agree_72b_stack_one_layer_per_call():
    # 64 Q / 8 KV heads, 256 tokens per frame: 64 row workgroups x 4 key ranges = 256
    # workgroups per one-layer launch (state full from frame 2 with capacity 512)
    _run_modes(WorkloadConfig("ks_72b_stack", 2, 64, 8, 128, 256, 4, 512, "bf16", "lowrank", 9202), True)
