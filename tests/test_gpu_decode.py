"""GPU parity of decoding over the detailed cache D (skv_decode_step) against the
fp64 oracle's decode_attention.

* After a StateKV stream of 12 frames at the 7B one-layer shape, decode calls of
  1, 3, 1, 8 and 64 tokens: every output against the oracle over all video
  tokens of D, the earlier decoded tokens and the new ones (causal); D's decode
  rows must hold the new tokens' K/V bytes.
* The 7B-shaped 28-layer stack with a 128-frame history (25,088 video tokens
  per KV head) written through the cache view, as the bench decodes it: two
  1-token calls, oracle on layers 0 and 27 (all 28 query heads).
* Error statuses: token counts out of range, more than max_decode_tokens, an
  fp32 context.

Tolerances: bf16 max-abs 2e-2, mean-abs 2e-3 (as every attention output here).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import statekv_oracle as orc
from paper_2605_31598_amd import FrameStepper, StateKVError
from paper_2605_31598_amd import binding as B
from workloads import CONFIGS
from workloads import generate as gen

from .gpu_harness import TOL_O, frame_tensors, say, to_device, widen

pytestmark = pytest.mark.gpu


def _bf16(rng, shape):
    return gen.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32))


def _decode_inputs(rng, L, wl, t):
    q = _bf16(rng, (L, wl.n_q_heads, t, wl.head_dim))
    k = _bf16(rng, (L, wl.n_kv_heads, t, wl.head_dim))
    v = _bf16(rng, (L, wl.n_kv_heads, t, wl.head_dim))
    return q, k, v


def _check(got, want, where):
    o_max, o_mean = TOL_O["bf16"]
    err = np.abs(got - want)
    assert err.max() <= o_max, f"{where}: max-abs {err.max():.3e}"
    assert err.mean() <= o_mean, f"{where}: mean-abs {err.mean():.3e}"
    return float(err.max())


def test_decode_after_a_statekv_stream_one_layer():
    wl = CONFIGS["vlm7b_1layer"]
    n_frames = 12
    chunks = [1, 3, 1, 8, 64]
    st = FrameStepper.from_workload(wl, max_frames=n_frames, max_decode_tokens=sum(chunks))
    rng = np.random.default_rng(5)
    try:
        out = torch.empty((1, wl.n_q_heads, wl.tokens_per_frame, wl.head_dim), dtype=torch.bfloat16, device="cuda")
        for n in range(n_frames):
            q, k, v, _ = frame_tensors(wl, n, [0])
            st.step(q, k, v, out)
        hist_k = np.concatenate([gen.frame_inputs(wl, 0, f)["k"] for f in range(n_frames)], axis=1)
        hist_v = np.concatenate([gen.frame_inputs(wl, 0, f)["v"] for f in range(n_frames)], axis=1)
        for t in chunks:
            q, k, v = _decode_inputs(rng, 1, wl, t)
            o = torch.empty((1, wl.n_q_heads, t, wl.head_dim), dtype=torch.bfloat16, device="cuda")
            say(f"decode {t} tokens after {hist_k.shape[1]} keys")
            st.decode(to_device(q, "bf16"), to_device(k, "bf16"), to_device(v, "bf16"), o)
            torch.cuda.synchronize()
            want = orc.decode_attention(widen(q[0], "bf16"), widen(hist_k, "bf16"), widen(hist_v, "bf16"),
                                        widen(k[0], "bf16"), widen(v[0], "bf16"), wl.scale)
            _check(o[0].float().cpu().numpy().astype(np.float64), want, f"decode t={t}")
            hist_k = np.concatenate([hist_k, k[0]], axis=1)
            hist_v = np.concatenate([hist_v, v[0]], axis=1)
        dk, dv = st.read_decode_rows(0)
        n_video = n_frames * wl.tokens_per_frame
        assert np.array_equal(dk, hist_k[:, n_video:]) and np.array_equal(dv, hist_v[:, n_video:])
    finally:
        st.close()


def test_decode_7b_stack_after_128_frames():
    wl = CONFIGS["vlm7b_28layer"]
    n = 128
    layers = [0, 27]
    st = FrameStepper.from_workload(wl, max_frames=n + 1, max_decode_tokens=4)
    rng = np.random.default_rng(6)
    try:
        hist = {}
        for l in layers:
            ks = np.concatenate([gen.frame_inputs(wl, l, f)["k"] for f in range(n)], axis=1)
            vs = np.concatenate([gen.frame_inputs(wl, l, f)["v"] for f in range(n)], axis=1)
            st.write_cache(l, ks, vs)
            hist[l] = [ks, vs]
        st.seek(n)
        L = wl.n_layers
        for call in range(2):
            q, k, v = _decode_inputs(rng, L, wl, 1)
            o = torch.empty((L, wl.n_q_heads, 1, wl.head_dim), dtype=torch.bfloat16, device="cuda")
            say(f"decode call {call}: 1 token over {n * wl.tokens_per_frame + call} cached tokens, 28 layers")
            st.decode(to_device(q, "bf16"), to_device(k, "bf16"), to_device(v, "bf16"), o)
            torch.cuda.synchronize()
            got = o.float().cpu().numpy().astype(np.float64)
            for l in layers:
                ks, vs = hist[l]
                want = orc.decode_attention(widen(q[l], "bf16"), widen(ks, "bf16"), widen(vs, "bf16"),
                                            widen(k[l], "bf16"), widen(v[l], "bf16"), wl.scale)
                e = _check(got[l], want, f"call {call} layer {l}")
                say(f"  layer {l}: max-abs {e:.2e}")
                hist[l] = [np.concatenate([ks, k[l]], axis=1), np.concatenate([vs, v[l]], axis=1)]
    finally:
        st.close()


def test_decode_error_statuses():
    wl = CONFIGS["vlm7b_1layer"].with_(capacity=64)
    st = FrameStepper.from_workload(wl, max_frames=4, max_decode_tokens=4)
    try:
        d, Hq, Hkv = wl.head_dim, wl.n_q_heads, wl.n_kv_heads

        def dec(t):
            q = torch.zeros((1, Hq, t, d), dtype=torch.bfloat16, device="cuda")
            k = torch.zeros((1, Hkv, t, d), dtype=torch.bfloat16, device="cuda")
            return q, k, k.clone(), torch.empty_like(q)

        lib = B.load_library()
        q, k, v, o = dec(1)
        assert lib.skv_decode_step(st.ctx, 0, 1, 0, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                   o.data_ptr()) == B.SKV_ERR_INVALID_ARG
        assert lib.skv_decode_step(st.ctx, 0, 1, 65, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                   o.data_ptr()) == B.SKV_ERR_INVALID_ARG
        assert lib.skv_decode_step(st.ctx, 0, 1, 1, q.data_ptr(), k.data_ptr() + 8, v.data_ptr(),
                                   o.data_ptr()) == B.SKV_ERR_INVALID_ARG  # misaligned key pointer
        q5, k5, v5, o5 = dec(5)
        with pytest.raises(StateKVError, match="CAPACITY"):
            st.decode(q5, k5, v5, o5)
        st.decode(q, k, v, o)  # a valid call still works after the refused ones
        torch.cuda.synchronize()
    finally:
        st.close()
    f32 = CONFIGS["tiny_f32"]
    st = FrameStepper.from_workload(f32, max_decode_tokens=2)
    try:
        q = torch.zeros((1, f32.n_q_heads, 1, f32.head_dim), dtype=torch.float32, device="cuda")
        k = torch.zeros((1, f32.n_kv_heads, 1, f32.head_dim), dtype=torch.float32, device="cuda")
        with pytest.raises(StateKVError, match="UNSUPPORTED"):
            st.decode(q, k, k.clone(), torch.empty_like(q))
    finally:
        st.close()
