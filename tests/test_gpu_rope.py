"""GPU parity of RoPE / YaRN at virtual positions, fused into the step, against the
fp64 oracle (rope_rotate: half-split pairs, rotated activations rounded to the
model dtype).

* StateKV streams with a non-zero position offset: the fp32 tiny shape with plain
  RoPE (scalar kernel) and the 7B one-layer shape with YaRN (MFMA kernel).  Every
  frame is compared with the oracle run on the GPU's own state entering it:
  outputs, scores (1e-3 relative), the selection rule on the GPU's scores
  (exact), and the rotated keys the state admits and the cache receives
  (within one unit in the last place of the model dtype: the oracle rounds an
  fp64 rotation, the kernels an fp32 one).
* Full SA and then decoding over the cache with RoPE: frame outputs, then
  decoded tokens whose positions continue the virtual length.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import statekv_oracle as orc
from paper_2605_31598_amd import FrameStepper
from workloads import CONFIGS
from workloads import generate as gen

from .gpu_harness import SCORE_REL, TOL_O, frame_tensors, gpu_state_as_oracle, say, to_device, widen

pytestmark = pytest.mark.gpu


def _ulp_close(got, want, dtype):
    """|got - want| <= one unit in the last place of the storage dtype at want, plus the
    fp32 rounding of the rotation's two products (2^-20 of the row's largest magnitude),
    which dominates where the two products cancel."""
    bits = 8 if dtype == "bf16" else 24
    _, e = np.frexp(want)
    ulp = np.ldexp(1.0, e - bits)
    slack = np.ldexp(np.abs(want).max(axis=-1, keepdims=True), -20)
    return np.all(np.abs(got - want) <= ulp + slack)


def _stream_rope(wl, n_frames, rope_kw, spec, policy="statekv", max_decode_tokens=0):
    """Streams n_frames, checking each against the oracle; returns the open stepper and
    the keys/values the cache holds (as fp64)."""
    st = FrameStepper.from_workload(wl, max_frames=n_frames, policy=policy, max_decode_tokens=max_decode_tokens,
                                    **rope_kw)
    out = torch.empty((1, wl.n_q_heads, wl.tokens_per_frame, wl.head_dim),
                      dtype=torch.bfloat16 if wl.dtype == "bf16" else torch.float32, device="cuda")
    full_k, full_v = [], []
    try:
        for n in range(n_frames):
            gpu_state = st.read_state(0)
            if policy == "full":
                state = orc.LayerState(
                    np.tile(wl.pos_offset + np.arange(n * wl.tokens_per_frame), (wl.n_kv_heads, 1)),
                    np.concatenate(full_k, axis=1) if n else np.zeros((wl.n_kv_heads, 0, wl.head_dim)),
                    np.concatenate(full_v, axis=1) if n else np.zeros((wl.n_kv_heads, 0, wl.head_dim)),
                    np.zeros((wl.n_kv_heads, n * wl.tokens_per_frame)))
            else:
                state = gpu_state_as_oracle(gpu_state, wl.dtype)
            q, k, v, host = frame_tensors(wl, n, [0])
            st.step(q, k, v, out)
            torch.cuda.synchronize()
            x = host[0]
            r = orc.frame_step(state, widen(x["q"], wl.dtype), widen(x["k"], wl.dtype), widen(x["v"], wl.dtype), n,
                               wl.capacity, wl.scale, wl.pos_offset, policy=policy, rope=spec)
            got = out[0].float().cpu().numpy().astype(np.float64)
            o_max, o_mean = TOL_O[wl.dtype]
            err = np.abs(got - r.out)
            assert err.max() <= o_max and err.mean() <= o_mean, f"frame {n}: output {err.max():.3e}/{err.mean():.3e}"
            ck, cv, _ = st.read_cache(0)
            T = wl.tokens_per_frame
            new_k = widen(ck[:, n * T:(n + 1) * T], wl.dtype)
            assert _ulp_close(new_k, r.k_stored, wl.dtype), f"frame {n}: rotated keys in the cache"
            assert np.array_equal(cv[:, n * T:(n + 1) * T], x["v"]), f"frame {n}: values in the cache"
            full_k.append(new_k)
            full_v.append(widen(cv[:, n * T:(n + 1) * T], wl.dtype))
            if policy == "statekv":
                gs = st.read_state(0)
                rows = np.arange(wl.n_kv_heads)[:, None]
                po = np.argsort(gs["pool_pos"], axis=1)
                sc = gs["pool_score"][rows, po].astype(np.float64)
                rel = np.abs(sc - r.pool_score) / r.pool_score
                assert rel.max() <= SCORE_REL, f"frame {n}: scores {rel.max():.3e}"
                for g in range(wl.n_kv_heads):
                    keep = orc.select_top(sc[g], gs["pool_pos"][g][po[g]].astype(np.int64), wl.capacity)
                    assert np.array_equal(np.sort(gs["pool_pos"][g][po[g]][keep]), np.sort(gs["pos"][g]))
                # rows the state admitted from this frame are the rotated frame keys
                fpos = orc.frame_positions(n, T, wl.pos_offset)
                for g in range(wl.n_kv_heads):
                    adm = np.nonzero(gs["pos"][g] >= fpos[0])[0]
                    t_idx = gs["pos"][g][adm] - fpos[0]
                    assert _ulp_close(widen(gs["k"][g][adm], wl.dtype), r.k_stored[g][t_idx], wl.dtype)
            if n % 4 == 0:
                say(f"  {wl.name} {policy} rope frame {n}: max-abs {err.max():.2e}")
    except BaseException:
        st.close()
        raise
    return st, full_k, full_v


def test_rope_plain_tiny_f32_statekv():
    wl = CONFIGS["tiny_f32"].with_(pos_offset=300)
    spec = orc.rope_spec(wl.head_dim, 10000.0, dtype="f32")
    st, _, _ = _stream_rope(wl, wl.n_frames, dict(rope="plain", rope_theta=10000.0), spec)
    st.close()


def test_yarn_vlm7b_one_layer_statekv():
    wl = CONFIGS["vlm7b_1layer"].with_(pos_offset=1000)
    spec = orc.rope_spec(wl.head_dim, 1e6, "yarn", factor=4.0, orig_max=8192, dtype="bf16")
    st, _, _ = _stream_rope(wl, 14, dict(rope="yarn", rope_theta=1e6, rope_factor=4.0, rope_orig_max=8192), spec)
    st.close()


def test_rope_full_attention_then_decode():
    wl = CONFIGS["vlm7b_1layer"].with_(pos_offset=50)
    spec = orc.rope_spec(wl.head_dim, 1e6, dtype="bf16")
    n_frames = 6
    kw = dict(rope="plain", rope_theta=1e6)
    st, full_k, full_v = _stream_rope(wl, n_frames, kw, spec, policy="full", max_decode_tokens=8)
    try:
        hist_k = np.concatenate(full_k, axis=1)
        hist_v = np.concatenate(full_v, axis=1)
        rng = np.random.default_rng(11)
        pos = wl.pos_offset + n_frames * wl.tokens_per_frame
        for t in (1, 3):
            qd = gen.f32_to_bf16_bits(rng.standard_normal((1, wl.n_q_heads, t, wl.head_dim)).astype(np.float32))
            kd = gen.f32_to_bf16_bits(rng.standard_normal((1, wl.n_kv_heads, t, wl.head_dim)).astype(np.float32))
            vd = gen.f32_to_bf16_bits(rng.standard_normal((1, wl.n_kv_heads, t, wl.head_dim)).astype(np.float32))
            o = torch.empty((1, wl.n_q_heads, t, wl.head_dim), dtype=torch.bfloat16, device="cuda")
            st.decode(to_device(qd, "bf16"), to_device(kd, "bf16"), to_device(vd, "bf16"), o)
            torch.cuda.synchronize()
            positions = pos + np.arange(t)
            want = orc.decode_attention(widen(qd[0], "bf16"), hist_k, hist_v, widen(kd[0], "bf16"),
                                        widen(vd[0], "bf16"), wl.scale, rope=spec, positions=positions)
            err = np.abs(o[0].float().cpu().numpy().astype(np.float64) - want)
            assert err.max() <= TOL_O["bf16"][0] and err.mean() <= TOL_O["bf16"][1], f"decode t={t}: {err.max():.3e}"
            dk, dv = st.read_decode_rows(0)
            k_rot = orc.rope_rotate(widen(kd[0], "bf16"), positions, spec)
            assert _ulp_close(widen(dk[:, -t:], "bf16"), k_rot, "bf16"), "rotated decode keys in the cache"
            hist_k = np.concatenate([hist_k, widen(dk[:, -t:], "bf16")], axis=1)
            hist_v = np.concatenate([hist_v, widen(vd[0], "bf16")], axis=1)
            pos += t
    finally:
        st.close()


def test_yarn_stack_layer_by_layer_and_whole_stack_calls():
    """A three-layer stack with YaRN: frames 0-2 one call per layer (the real-model pattern),
    frame 3 one call for all layers, then decoding one layer per call.  Every call rotates
    its own layers' new keys; each layer is checked against the oracle on the GPU's state."""
    from workloads import WorkloadConfig

    wl = WorkloadConfig("yarn_stack", 3, 8, 2, 128, 24, 4, 40, "bf16", "iid", 5151, pos_offset=777)
    spec = orc.rope_spec(wl.head_dim, 1e6, "yarn", factor=4.0, orig_max=4096, dtype="bf16")
    st = FrameStepper.from_workload(wl, max_decode_tokens=4, rope="yarn", rope_theta=1e6, rope_factor=4.0,
                                    rope_orig_max=4096)
    T, L = wl.tokens_per_frame, wl.n_layers
    try:
        for n in range(wl.n_frames):
            states = {l: gpu_state_as_oracle(st.read_state(l), "bf16") for l in range(L)}
            q, k, v, host = frame_tensors(wl, n, list(range(L)))
            out = torch.empty((L, wl.n_q_heads, T, wl.head_dim), dtype=torch.bfloat16, device="cuda")
            if n < 3:
                for l in range(L):
                    st.step(q[l:l + 1], k[l:l + 1], v[l:l + 1], out[l:l + 1], layer_begin=l, layer_count=1)
            else:
                st.step(q, k, v, out)
            torch.cuda.synchronize()
            for l in range(L):
                x = host[l]
                r = orc.frame_step(states[l], widen(x["q"], "bf16"), widen(x["k"], "bf16"), widen(x["v"], "bf16"), n,
                                   wl.capacity, wl.scale, wl.pos_offset, rope=spec)
                err = np.abs(out[l].float().cpu().numpy().astype(np.float64) - r.out)
                assert err.max() <= TOL_O["bf16"][0] and err.mean() <= TOL_O["bf16"][1], \
                    f"frame {n} layer {l}: output {err.max():.3e}"
                ck, _, _ = st.read_cache(l)
                assert _ulp_close(widen(ck[:, n * T:(n + 1) * T], "bf16"), r.k_stored, "bf16"), \
                    f"frame {n} layer {l}: rotated keys in the cache"
        say(f"  yarn stack: {wl.n_frames} frames ok")
        rng = np.random.default_rng(5)
        t = 2
        pos = wl.pos_offset + wl.n_frames * T + np.arange(t)
        for l in range(L):
            qd = gen.f32_to_bf16_bits(rng.standard_normal((1, wl.n_q_heads, t, wl.head_dim)).astype(np.float32))
            kd = gen.f32_to_bf16_bits(rng.standard_normal((1, wl.n_kv_heads, t, wl.head_dim)).astype(np.float32))
            vd = gen.f32_to_bf16_bits(rng.standard_normal((1, wl.n_kv_heads, t, wl.head_dim)).astype(np.float32))
            ck, cv, _ = st.read_cache(l)
            o = torch.empty((1, wl.n_q_heads, t, wl.head_dim), dtype=torch.bfloat16, device="cuda")
            st.decode(to_device(qd, "bf16"), to_device(kd, "bf16"), to_device(vd, "bf16"), o, layer_begin=l,
                      layer_count=1)
            torch.cuda.synchronize()
            hist_k = widen(ck[:, :wl.n_frames * T], "bf16")
            hist_v = widen(cv[:, :wl.n_frames * T], "bf16")
            want = orc.decode_attention(widen(qd[0], "bf16"), hist_k, hist_v, widen(kd[0], "bf16"),
                                        widen(vd[0], "bf16"), wl.scale, rope=spec, positions=pos)
            err = np.abs(o[0].float().cpu().numpy().astype(np.float64) - want)
            assert err.max() <= TOL_O["bf16"][0] and err.mean() <= TOL_O["bf16"][1], f"decode layer {l}: {err.max():.3e}"
            dk, _ = st.read_decode_rows(l)
            assert _ulp_close(widen(dk[:, -t:], "bf16"), orc.rope_rotate(widen(kd[0], "bf16"), pos, spec), "bf16")
    finally:
        st.close()
