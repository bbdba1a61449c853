"""GPU parity of the two baseline policies against the fp64 oracle.

* SKV_POLICY_FULL (streaming full self-attention over the decode cache, the
  Full SA baseline): every frame's output equals the oracle's causal attention
  over all earlier tokens plus the frame; the cache holds the input rows; no
  state is kept.  Whole short videos at the small shapes, and one frame of the
  7B-shaped 28-layer stack at frame 100 (19,796 keys per query) on a cache
  written through the cache view, checked on the first and last layer.
* SKV_POLICY_RECENT (recency window): outputs against the oracle, and the state
  positions exactly the last min(B, seen) tokens, frame after frame.

Same tolerances as the StateKV parity tests (bf16 max-abs 2e-2 / mean-abs 2e-3,
fp32 1e-5); the recency window's informational scores within 1e-3 relative.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import statekv_oracle as orc
from paper_2605_31598_amd import FrameStepper
from workloads import CONFIGS
from workloads import generate as gen

from .gpu_harness import SCORE_REL, TOL_O, frame_tensors, say, to_device, widen

pytestmark = pytest.mark.gpu


def _oracle_frame(wl, state, raw, frame, policy):
    return orc.frame_step(state, widen(raw["q"], wl.dtype), widen(raw["k"], wl.dtype), widen(raw["v"], wl.dtype),
                          frame, wl.capacity, wl.scale, wl.pos_offset, policy=policy)


def _check_out(wl, got, want, where):
    o_max, o_mean = TOL_O[wl.dtype]
    err = np.abs(got - want)
    assert err.max() <= o_max, f"{where}: output max-abs {err.max():.3e} > {o_max}"
    assert err.mean() <= o_mean, f"{where}: output mean-abs {err.mean():.3e} > {o_mean}"
    return float(err.max())


def _stream(wl, policy, n_frames, layers):
    """Whole-stack calls on the GPU, oracle on `layers`; compares every frame."""
    st = FrameStepper.from_workload(wl, max_frames=n_frames, policy=policy)
    states = {l: orc.LayerState.empty(wl.n_kv_heads, wl.head_dim) for l in layers}
    out = torch.empty((wl.n_layers, wl.n_q_heads, wl.tokens_per_frame, wl.head_dim),
                      dtype=torch.bfloat16 if wl.dtype == "bf16" else torch.float32, device="cuda")
    worst = 0.0
    try:
        for n in range(n_frames):
            q, k, v, host = frame_tensors(wl, n, layers)
            st.step(q, k, v, out)
            torch.cuda.synchronize()
            got = out.float().cpu().numpy().astype(np.float64)
            for l in layers:
                r = _oracle_frame(wl, states[l], host[l], n, policy)
                worst = max(worst, _check_out(wl, got[l], r.out, f"{policy} frame {n} layer {l}"))
                gs = st.read_state(l)
                if policy == "full":
                    assert gs["size"] == 0
                else:
                    assert np.array_equal(np.sort(gs["pos"], axis=1), r.state.pos), f"frame {n} layer {l}: state"
                    po = np.argsort(gs["pool_pos"], axis=1)
                    rows = np.arange(wl.n_kv_heads)[:, None]
                    assert np.array_equal(gs["pool_pos"][rows, po], r.pool_pos)
                    rel = np.abs(gs["pool_score"][rows, po] - r.pool_score) / r.pool_score
                    assert rel.max() <= SCORE_REL, f"frame {n} layer {l}: score rel {rel.max():.3e}"
                states[l] = r.state
            if n % 4 == 0:
                say(f"  {wl.name} {policy} frame {n}: worst max-abs so far {worst:.2e}")
        for l in layers:
            ck, cv, nt = st.read_cache(l)
            assert nt == n_frames * wl.tokens_per_frame
            want_k = np.concatenate([gen.frame_inputs(wl, l, f)["k"] for f in range(n_frames)], axis=1)
            want_v = np.concatenate([gen.frame_inputs(wl, l, f)["v"] for f in range(n_frames)], axis=1)
            assert np.array_equal(ck, want_k) and np.array_equal(cv, want_v), f"layer {l}: decode cache bytes"
    finally:
        st.close()
    return worst


def test_full_policy_tiny_f32_whole_video():
    wl = CONFIGS["tiny_f32"]
    say(f"full: {wl.name}")
    _stream(wl, "full", wl.n_frames, [0])


def test_full_policy_vlm7b_one_layer_12_frames():
    wl = CONFIGS["vlm7b_1layer"]
    say(f"full: {wl.name}, 12 frames (up to 2352 keys)")
    _stream(wl, "full", 12, [0])


def test_recent_policy_tiny_f32_whole_video():
    wl = CONFIGS["tiny_f32"].with_(capacity=20)  # a window that is not a whole number of frames
    say(f"recent: {wl.name} B=20")
    _stream(wl, "recent", wl.n_frames, [0])


def test_recent_policy_vlm7b_one_layer():
    wl = CONFIGS["vlm7b_1layer"]
    say(f"recent: {wl.name}, 10 frames")
    _stream(wl, "recent", 10, [0])


def test_full_policy_7b_stack_at_frame_100():
    """One frame of the 28-layer stack with a 100-frame history in the cache (19,600
    cached tokens per KV head), as the bench times it; oracle on layers 0 and 27 for
    KV heads 0 and 3 (their 7 query heads each)."""
    wl = CONFIGS["vlm7b_28layer"]
    n = 100
    layers = [0, 27]
    heads = [0, 3]
    st = FrameStepper.from_workload(wl, max_frames=n + 1, policy="full")
    try:
        hist = {}
        for l in layers:
            ks = np.concatenate([gen.frame_inputs(wl, l, f)["k"] for f in range(n)], axis=1)
            vs = np.concatenate([gen.frame_inputs(wl, l, f)["v"] for f in range(n)], axis=1)
            st.write_cache(l, ks, vs)
            hist[l] = (ks, vs)
        st.seek(n)
        q, k, v, host = frame_tensors(wl, n, layers)
        out = torch.empty((wl.n_layers, wl.n_q_heads, wl.tokens_per_frame, wl.head_dim), dtype=torch.bfloat16,
                          device="cuda")
        say(f"full: {wl.name} frame {n}, {n * wl.tokens_per_frame} cached tokens")
        st.step(q, k, v, out)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy().astype(np.float64)
        G = wl.group
        for l in layers:
            ks, vs = hist[l]
            for g in heads:
                hs = slice(g * G, (g + 1) * G)
                k_pool = widen(np.concatenate([ks[g:g + 1], host[l]["k"][g:g + 1]], axis=1), wl.dtype)
                v_pool = widen(np.concatenate([vs[g:g + 1], host[l]["v"][g:g + 1]], axis=1), wl.dtype)
                o, _ = orc.frame_attention(widen(host[l]["q"][hs], wl.dtype), k_pool, v_pool, ks.shape[1], wl.scale)
                e = _check_out(wl, got[l, hs], o, f"full frame {n} layer {l} kv head {g}")
                say(f"  layer {l} kv head {g}: max-abs {e:.2e}")
        ck, cv, nt = st.read_cache(27)
        assert nt == (n + 1) * wl.tokens_per_frame
        assert np.array_equal(ck[:, n * wl.tokens_per_frame:], host[27]["k"])
    finally:
        st.close()
