"""Shared machinery of the GPU parity tests: run the library's frame step and
the fp64 oracle on the same seeded inputs and compare.

Acceptance (per frame):
* attention output: bf16 max-abs <= 2e-2 and mean-abs <= 2e-3; fp32 max-abs <= 1e-5;
* importance scores of every candidate: relative error <= 1e-3;
* selected positions: identical to the oracle's, except at a near-tie (the
  oracle's B-th and (B+1)-th scores differ by less than 1e-4 relative), which
  is counted and reported instead;
* selected positions: identical, with no exception, to the oracle's selection
  rule applied to the GPU's own fp32 scores (the decision taken in one precision);
* state and decode-cache rows: byte-identical to the input rows.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import statekv_oracle as orc
from paper_2605_31598_amd import FrameStepper
from workloads import generate as gen

TOL_O = {"bf16": (2e-2, 2e-3), "f32": (1e-5, 1e-5)}
SCORE_REL = 1e-3
NEAR_TIE_REL = 1e-4


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(arr, dtype):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def widen(arr, dtype):
    return gen.to_f64(arr, dtype)


def gpu_state_as_oracle(st, dtype):
    """GPU slots (any order) -> oracle LayerState in ascending position."""
    order = np.argsort(st["pos"], axis=1, kind="stable")
    rows = np.arange(st["pos"].shape[0])[:, None]
    return orc.LayerState(pos=st["pos"][rows, order].astype(np.int64), k=widen(st["k"][rows, order], dtype),
                          v=widen(st["v"][rows, order], dtype), score=st["score"][rows, order].astype(np.float64))


def oracle_state_bytes(state, dtype):
    """Oracle state (fp64 values that came from dtype inputs) -> storage arrays for the GPU."""
    if dtype == "bf16":
        k = gen.f32_to_bf16_bits(state.k.astype(np.float32))
        v = gen.f32_to_bf16_bits(state.v.astype(np.float32))
    else:
        k = state.k.astype(np.float32)
        v = state.v.astype(np.float32)
    return state.pos.astype(np.int32), k, v


def near_tie(scores, capacity):
    """True when the oracle's capacity-th and next score are within NEAR_TIE_REL."""
    if scores.shape[0] <= capacity or capacity == 0:
        return False
    s = np.sort(scores)[::-1]
    a, b = s[capacity - 1], s[capacity]
    return (a - b) <= NEAR_TIE_REL * abs(a)


def compare_step(res, out_gpu, pool_gpu_score, pool_gpu_pos, kept_gpu_pos, capacity, dtype, where):
    """Compare one layer-frame; returns a report dict, raises AssertionError on failure."""
    rep = {"where": where}
    o_max, o_mean = TOL_O[dtype]
    err = np.abs(out_gpu - res.out)
    rep["o_max"], rep["o_mean"] = float(err.max()), float(err.mean())
    assert rep["o_max"] <= o_max, f"{where}: output max-abs {rep['o_max']:.3e} > {o_max}"
    assert rep["o_mean"] <= o_mean, f"{where}: output mean-abs {rep['o_mean']:.3e} > {o_mean}"

    H = res.pool_pos.shape[0]
    rel_max, n_tie, n_setdiff = 0.0, 0, 0
    for g in range(H):
        go = np.argsort(pool_gpu_pos[g], kind="stable")
        oo = np.argsort(res.pool_pos[g], kind="stable")
        gp, op = pool_gpu_pos[g][go], res.pool_pos[g][oo]
        assert np.array_equal(gp, op), f"{where}: candidate positions differ (kv head {g})"
        gs, os_ = pool_gpu_score[g][go].astype(np.float64), res.pool_score[g][oo]
        rel = np.abs(gs - os_) / np.abs(os_)
        rel_max = max(rel_max, float(rel.max()))
        # same-precision rule: the oracle's selection applied to the GPU's own scores
        own = orc.select_top(gs, gp.astype(np.int64), capacity)
        own_pos = np.sort(gp[own])
        kg = np.sort(kept_gpu_pos[g])
        assert np.array_equal(own_pos, kg), f"{where}: GPU selection is not Top-B of its own scores (kv head {g})"
        ko = np.sort(res.state.pos[g])
        if not np.array_equal(ko, kg):
            if near_tie(res.pool_score[g], capacity):
                n_tie += 1
            else:
                n_setdiff += 1
    rep["score_rel_max"] = rel_max
    rep["near_tie_diffs"] = n_tie
    assert rel_max <= SCORE_REL, f"{where}: score relative error {rel_max:.3e} > {SCORE_REL}"
    assert n_setdiff == 0, f"{where}: selected set differs from the oracle's away from a near-tie ({n_setdiff} heads)"
    return rep


def frame_tensors(wl, frame, layers, L=None):
    """Device q, k, v for all L layers of one frame: generator values on `layers`, zeros elsewhere.
    Returns (q, k, v, host dict layer -> raw inputs)."""
    L = wl.n_layers if L is None else L
    Hq, Hkv, T, d = wl.n_q_heads, wl.n_kv_heads, wl.tokens_per_frame, wl.head_dim
    npdt = np.uint16 if wl.dtype == "bf16" else np.float32
    q = np.zeros((L, Hq, T, d), dtype=npdt)
    k = np.zeros((L, Hkv, T, d), dtype=npdt)
    v = np.zeros((L, Hkv, T, d), dtype=npdt)
    host = {}
    for l in layers:
        x = gen.frame_inputs(wl, l, frame)
        q[l], k[l], v[l] = x["q"], x["k"], x["v"]
        host[l] = x
    return to_device(q, wl.dtype), to_device(k, wl.dtype), to_device(v, wl.dtype), host


def oracle_step(wl, state, raw, frame):
    return orc.frame_step(state, widen(raw["q"], wl.dtype), widen(raw["k"], wl.dtype), widen(raw["v"], wl.dtype),
                          frame, wl.capacity, wl.scale, wl.pos_offset)


def run_tracking(wl, n_frames, layers, start_frame=0, forced=None, independent=True, log_every=1, per_layer=False):
    """Stream frames through the GPU (all layers per call, or one call per layer
    with `per_layer`, the real-model calling pattern).  Every frame and every
    checked layer is compared with the oracle run on the GPU's own state entering
    that frame (so a near-tie cannot derail later frames).  With `independent`, the
    oracle also evolves its own state, and the first frame where the two states
    differ is reported.  Returns a summary dict."""
    stepper = FrameStepper.from_workload(wl, max_frames=start_frame + n_frames)
    L = wl.n_layers
    summary = {"frames": n_frames, "layers": list(layers), "near_tie_diffs": 0, "o_max": 0.0, "o_mean": 0.0,
               "score_rel_max": 0.0, "first_divergence": None}
    own = {l: orc.LayerState.empty(wl.n_kv_heads, wl.head_dim) for l in layers}
    try:
        if start_frame:
            stepper.seek(start_frame)
        if forced:
            for l, st in forced.items():
                pos, kb, vb = oracle_state_bytes(st, wl.dtype)
                stepper.write_state(l, pos, kb, vb)
                own[l] = st.copy()
        out = torch.empty((L, wl.n_q_heads, wl.tokens_per_frame, wl.head_dim),
                          dtype=torch.bfloat16 if wl.dtype == "bf16" else torch.float32, device="cuda")
        for n in range(start_frame, start_frame + n_frames):
            q, k, v, host = frame_tensors(wl, n, layers)
            before = {l: gpu_state_as_oracle(stepper.read_state(l), wl.dtype) for l in layers}
            if n % log_every == 0:
                say(f"  [{wl.name}] frame {n} (state {before[layers[0]].size}) layers {list(layers)}")
            if per_layer:
                for l in range(L):
                    stepper.step(q[l:l + 1], k[l:l + 1], v[l:l + 1], out[l:l + 1], layer_begin=l, layer_count=1)
            else:
                stepper.step(q, k, v, out)
            out_h = out.float().cpu().numpy().astype(np.float64)
            for l in layers:
                res = oracle_step(wl, before[l], host[l], n)
                after = stepper.read_state(l)
                rep = compare_step(res, out_h[l], after["pool_score"], after["pool_pos"], after["pos"],
                                   wl.capacity, wl.dtype, f"{wl.name} layer {l} frame {n}")
                # state rows are the input bytes
                st_after = gpu_state_as_oracle(after, wl.dtype)
                pool_k = np.concatenate([before[l].k, widen(host[l]["k"], wl.dtype)], axis=1)
                pool_p = res.pool_pos
                for g in range(wl.n_kv_heads):
                    idx = np.searchsorted(pool_p[g], st_after.pos[g]) if np.all(np.diff(pool_p[g]) > 0) else None
                    if idx is not None:
                        assert np.array_equal(st_after.k[g], pool_k[g][idx]), f"state rows changed, layer {l} frame {n}"
                summary["near_tie_diffs"] += rep["near_tie_diffs"]
                for key in ("o_max", "o_mean", "score_rel_max"):
                    summary[key] = max(summary[key], rep[key])
                if independent:
                    r_own = oracle_step(wl, own[l], host[l], n)
                    own[l] = r_own.state
                    if summary["first_divergence"] is None and not np.array_equal(np.sort(r_own.state.pos, axis=1),
                                                                                np.sort(after["pos"], axis=1)):
                        summary["first_divergence"] = n
        # decode cache holds every frame's rows, byte for byte
        for l in layers:
            ck, cv, n_tok = stepper.read_cache(l)
            assert n_tok == (start_frame + n_frames) * wl.tokens_per_frame
            for n in range(start_frame, start_frame + n_frames):
                x = gen.frame_inputs(wl, l, n)
                rows = slice(n * wl.tokens_per_frame, (n + 1) * wl.tokens_per_frame)
                assert np.array_equal(ck[:, rows], x["k"]), f"decode cache K differs, layer {l} frame {n}"
                assert np.array_equal(cv[:, rows], x["v"]), f"decode cache V differs, layer {l} frame {n}"
    finally:
        stepper.close()
    return summary


def recent_state(wl, layer, frame):
    """A valid full state entering `frame`: the most recent min(B, frame*T) tokens, as oracle state."""
    T, B = wl.tokens_per_frame, wl.capacity
    S = wl.state_size(frame)
    first = frame * T - S
    frames = range(first // T, frame)
    ks, vs, ps = [], [], []
    for f in frames:
        x = gen.frame_inputs(wl, layer, f)
        ks.append(x["k"])
        vs.append(x["v"])
        ps.append(orc.frame_positions(f, T, wl.pos_offset))
    k = np.concatenate(ks, axis=1)[:, -S:] if S else np.zeros((wl.n_kv_heads, 0, wl.head_dim))
    v = np.concatenate(vs, axis=1)[:, -S:] if S else np.zeros((wl.n_kv_heads, 0, wl.head_dim))
    p = np.concatenate(ps)[-S:] if S else np.zeros(0, dtype=np.int64)
    H = wl.n_kv_heads
    return orc.LayerState(pos=np.tile(p, (H, 1)), k=widen(k, wl.dtype), v=widen(v, wl.dtype), score=np.zeros((H, S)))
