"""Deferred selection of one-layer calls, through the C ABI.

A call that covers part of a multi-layer stack with a key-split attention plan
(one layer of the 7B shape) leaves its selection and state update to the output
launch of the next such call on other layers, or to the next use of the state.
Every result must equal that of a context that never defers (split_refresh = 1:
selection, update and append as launches of their own in the same call), bit
for bit: each call's attention output, and after every frame (and in the middle
of one) every layer's state slots, positions, scores, candidate pool and
decode-cache rows.  The caller's k and v buffers are reused for every call, so
a deferred update that read them instead of the decode cache would copy the
wrong layer's rows.  Covered: StateKV with and without YaRN, the recency window,
a whole-stack call between one-layer calls, a state read in the middle of a
frame, and a reset with a selection still deferred.
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


def _same_state(a, b, layers, where):
    for l in layers:
        x, y = a.read_state(l), b.read_state(l)
        assert x["size"] == y["size"], f"{where}: state size of layer {l}"
        for key in ("pos", "score", "k", "v", "pool_score", "pool_pos"):
            assert np.array_equal(x[key], y[key]), f"{where}: {key} of layer {l}"
        ca, cb = a.read_cache(l), b.read_cache(l)
        assert ca[2] == cb[2] and np.array_equal(ca[0], cb[0]) and np.array_equal(ca[1], cb[1]), \
            f"{where}: decode cache of layer {l}"


def _stream(wl, n_frames, whole_stack_frames=(), mid_read=None, pair=None, last_check=True, **kw):
    """Steps a deferring and a non-deferring context (new ones, or `pair`) through
    n_frames frames, one layer per call except on whole_stack_frames; compares
    outputs per call, states after every third frame (reading a state enqueues a
    deferred selection, so the frames in between carry the last layer's selection
    into the next frame's first call) and after the last frame unless last_check
    is False, and the state of layer mid_read[1] after its call in frame
    mid_read[0]."""
    L, Hq, Hkv, T, d = wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.tokens_per_frame, wl.head_dim
    if pair is None:
        pair = (FrameStepper.from_workload(wl, **kw), FrameStepper.from_workload(wl, split_refresh=True, **kw))
    dfr, ref = pair
    try:
        bufs = {}
        for name, st in (("dfr", dfr), ("ref", ref)):  # reused by every call of that context
            bufs[name] = (torch.empty((L, Hq, T, d), dtype=torch.bfloat16, device="cuda"),
                          torch.empty((L, Hkv, T, d), dtype=torch.bfloat16, device="cuda"),
                          torch.empty((L, Hkv, T, d), dtype=torch.bfloat16, device="cuda"),
                          torch.empty((L, Hq, T, d), dtype=torch.bfloat16, device="cuda"))
        for n in range(n_frames):
            q, k, v, _ = frame_tensors(wl, n, list(range(L)))
            spans = [(0, L)] if n in whole_stack_frames else [(l, 1) for l in range(L)]
            for l0, lc in spans:
                sl = slice(0, lc)
                outs = []
                for name, st in (("dfr", dfr), ("ref", ref)):
                    qb, kb, vb, ob = bufs[name]
                    qb[sl].copy_(q[l0:l0 + lc])
                    kb[sl].copy_(k[l0:l0 + lc])
                    vb[sl].copy_(v[l0:l0 + lc])
                    st.step(qb[sl], kb[sl], vb[sl], ob[sl], layer_begin=l0, layer_count=lc)
                    outs.append(ob[sl].clone())
                assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16)), \
                    f"{wl.name} frame {n} layers {l0}..{l0 + lc - 1}: output"
                if mid_read is not None and (n, l0) == mid_read:
                    _same_state(dfr, ref, [l0], f"{wl.name} frame {n}, after layer {l0}")
            if n % 3 == 2 or (last_check and n == n_frames - 1):
                _same_state(dfr, ref, range(L), f"{wl.name} frame {n}")
        return dfr, ref
    except BaseException:
        dfr.close()
        ref.close()
        raise


def _wl(name, seed, layers=3, frames=10):
    # 7B-shaped layers (28 Q / 4 KV heads, d 128, 196 tokens per frame): a one-layer
    # call splits the keys; capacity 1024 is full from frame 6 on
    return WorkloadConfig(name, layers, 28, 4, 128, 196, frames, 1024, "bf16", "iid", seed)


def test_deferred_selection_matches_undeferred_statekv():
    wl = _wl("deferred_7b", 9100)
    dfr, ref = _stream(wl, wl.n_frames, whole_stack_frames=(7,), mid_read=(9, 1), last_check=False)
    say(f"{wl.name}: {wl.n_frames} frames equal (one whole-stack frame, one mid-frame read)")
    # a new video on the same contexts: the reset comes while the last layer's
    # selection of the last frame is still deferred, and drops it
    for st in (dfr, ref):
        st.reset()
    dfr, ref = _stream(wl, 3, pair=(dfr, ref))
    dfr.close()
    ref.close()
    say(f"{wl.name}: equal again after a reset")


def test_deferred_selection_matches_undeferred_yarn():
    wl = _wl("deferred_7b_yarn", 9101, layers=2, frames=8)
    dfr, ref = _stream(wl, wl.n_frames, rope="yarn", rope_theta=1e6, rope_factor=4.0, rope_orig_max=4096)
    dfr.close()
    ref.close()
    say(f"{wl.name}: {wl.n_frames} frames equal with YaRN")


def test_deferred_selection_matches_undeferred_recent():
    wl = _wl("deferred_7b_recent", 9102, layers=2, frames=8)
    dfr, ref = _stream(wl, wl.n_frames, policy="recent")
    dfr.close()
    ref.close()
    say(f"{wl.name}: {wl.n_frames} frames equal under the recency window")
