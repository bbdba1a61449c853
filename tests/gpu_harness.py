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


def straddling_tie(scores, capacity):
    """True when entries exactly equal to the capacity-th largest score fall on both sides
    of the boundary (some kept, some not): the tie rule (lowest position) decides them."""
    if scores.shape[0] <= capacity or capacity == 0:
        return False
    s = np.sort(scores)[::-1]
    thr = s[capacity - 1]
    above = int((scores > thr).sum())
    equal = int((scores == thr).sum())
    return above + equal > capacity


def boundary_gap(scores, capacity):
    """Relative gap between the capacity-th and the next largest score (inf if no pruning)."""
    if scores.shape[0] <= capacity or capacity == 0:
        return float("inf")
    s = np.sort(scores)[::-1]
    a, b = s[capacity - 1], s[capacity]
    return float((a - b) / abs(a)) if a != 0 else 0.0


def compare_step(res, out_gpu, pool_gpu_score, pool_gpu_pos, kept_gpu_pos, capacity, dtype, where):
    """Compare one layer-frame; returns a report dict, raises AssertionError on failure.

    Report fields: output errors, the largest score error, and per KV head whose GPU
    selection differs from the oracle's (a near-tie, else a failure) the oracle's
    boundary gap; the number of heads whose oracle / GPU scores have exact ties
    straddling the capacity boundary."""
    rep = {"where": where}
    o_max, o_mean = TOL_O[dtype]
    err = np.abs(out_gpu - res.out)
    rep["o_max"], rep["o_mean"] = float(err.max()), float(err.mean())
    assert rep["o_max"] <= o_max, f"{where}: output max-abs {rep['o_max']:.3e} > {o_max}"
    assert rep["o_mean"] <= o_mean, f"{where}: output mean-abs {rep['o_mean']:.3e} > {o_mean}"

    H = res.pool_pos.shape[0]
    rel_max, n_setdiff = 0.0, 0
    rep["diverged_heads"] = []
    rep["straddle_oracle"] = rep["straddle_gpu"] = 0
    for g in range(H):
        go = np.argsort(pool_gpu_pos[g], kind="stable")
        oo = np.argsort(res.pool_pos[g], kind="stable")
        gp, op = pool_gpu_pos[g][go], res.pool_pos[g][oo]
        assert np.array_equal(gp, op), f"{where}: candidate positions differ (kv head {g})"
        gs, os_ = pool_gpu_score[g][go].astype(np.float64), res.pool_score[g][oo]
        rel = np.abs(gs - os_) / np.abs(os_)
        rel_max = max(rel_max, float(rel.max()))
        rep["straddle_oracle"] += int(straddling_tie(os_, capacity))
        rep["straddle_gpu"] += int(straddling_tie(gs, capacity))
        # same-precision rule: the oracle's selection applied to the GPU's own scores
        own = orc.select_top(gs, gp.astype(np.int64), capacity)
        own_pos = np.sort(gp[own])
        kg = np.sort(kept_gpu_pos[g])
        assert np.array_equal(own_pos, kg), f"{where}: GPU selection is not Top-B of its own scores (kv head {g})"
        ko = np.sort(res.state.pos[g])
        if not np.array_equal(ko, kg):
            gap = boundary_gap(res.pool_score[g], capacity)
            if near_tie(res.pool_score[g], capacity):
                rep["diverged_heads"].append((g, gap))
            else:
                n_setdiff += 1
    rep["score_rel_max"] = rel_max
    rep["near_tie_diffs"] = len(rep["diverged_heads"])
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


def _check_state_rows(before, raw, res, after_raw, dtype, where):
    """Every state slot holds, byte for byte, the K and V row of the candidate whose
    position it reports (a state entry's or a frame token's input row)."""
    H = res.pool_pos.shape[0]
    stored = (np.concatenate([oracle_state_bytes(before, dtype)[1], raw["k"]], axis=1),
              np.concatenate([oracle_state_bytes(before, dtype)[2], raw["v"]], axis=1))
    for g in range(H):
        pool_p = res.pool_pos[g]
        assert np.all(np.diff(pool_p) > 0), f"{where}: pool positions not ascending (kv head {g})"
        idx = np.searchsorted(pool_p, after_raw["pos"][g])
        assert np.array_equal(pool_p[idx], after_raw["pos"][g]), f"{where}: unknown state position (kv head {g})"
        assert np.array_equal(after_raw["k"][g], stored[0][g][idx]), f"{where}: state K rows changed (kv head {g})"
        assert np.array_equal(after_raw["v"][g], stored[1][g][idx]), f"{where}: state V rows changed (kv head {g})"


def run_tracking(wl, n_frames, layers, start_frame=0, forced=None, log_every=1, per_layer=False):
    """Stream frames through the GPU, end to end and unforced after `start_frame`
    (all layers per call, or one call per layer with `per_layer`, the real-model
    calling pattern); layers outside `layers` get zero inputs.

    Every frame of every checked layer is compared with the oracle run on the
    GPU's state entering it.  From the empty state (or a forced one) that state
    is the oracle's own evolution (Eq. 6 applied frame after frame) until a frame
    where the GPU keeps a different set; such a frame must be a near-tie for that
    KV head (asserted in compare_step) and is recorded in `divergences` with the
    oracle's boundary gap; the oracle then follows the GPU's equally valid choice.
    Also checked every frame: state K and V rows and the frame's decode-cache rows
    are the input bytes.  Returns a summary dict."""
    import concurrent.futures as cf

    stepper = FrameStepper.from_workload(wl, max_frames=start_frame + n_frames)
    L, T = wl.n_layers, wl.tokens_per_frame
    summary = {"frames": n_frames, "layers": list(layers), "near_tie_diffs": 0, "o_max": 0.0, "o_mean": 0.0,
               "score_rel_max": 0.0, "first_divergence": None, "divergences": [], "straddle_oracle": 0,
               "straddle_gpu": 0}
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    pool = cf.ThreadPoolExecutor(max_workers=max(1, len(layers)))
    try:
        if start_frame:
            stepper.seek(start_frame)
        if forced:
            for l, st in forced.items():
                pos, kb, vb = oracle_state_bytes(st, wl.dtype)
                stepper.write_state(l, pos, kb, vb)
        q_dev = torch.zeros((L, wl.n_q_heads, T, wl.head_dim), dtype=tdt, device="cuda")
        k_dev = torch.zeros((L, wl.n_kv_heads, T, wl.head_dim), dtype=tdt, device="cuda")
        v_dev = torch.zeros_like(k_dev)
        out = torch.empty_like(q_dev)
        before = {l: gpu_state_as_oracle(stepper.read_state(l), wl.dtype) for l in layers}
        for n in range(start_frame, start_frame + n_frames):
            host = dict(zip(layers, pool.map(lambda l: gen.frame_inputs(wl, l, n), layers)))
            for l in layers:
                q_dev[l].copy_(to_device(host[l]["q"], wl.dtype))
                k_dev[l].copy_(to_device(host[l]["k"], wl.dtype))
                v_dev[l].copy_(to_device(host[l]["v"], wl.dtype))
            if n % log_every == 0:
                say(f"  [{wl.name}] frame {n} (state {before[layers[0]].size}) layers {list(layers)}")
            if per_layer:
                for l in range(L):
                    stepper.step(q_dev[l:l + 1], k_dev[l:l + 1], v_dev[l:l + 1], out[l:l + 1], layer_begin=l,
                                 layer_count=1)
            else:
                stepper.step(q_dev, k_dev, v_dev, out)
            out_h = {l: out[l].float().cpu().numpy().astype(np.float64) for l in layers}
            results = dict(zip(layers, pool.map(lambda l: oracle_step(wl, before[l], host[l], n), layers)))
            for l in layers:
                res = results[l]
                where = f"{wl.name} layer {l} frame {n}"
                after = stepper.read_state(l)
                rep = compare_step(res, out_h[l], after["pool_score"], after["pool_pos"], after["pos"],
                                   wl.capacity, wl.dtype, where)
                _check_state_rows(before[l], host[l], res, after, wl.dtype, where)
                # the frame's rows of the decode cache
                ck, cv, n_tok = stepper.read_cache_rows(l, n * T, (n + 1) * T)
                assert n_tok == (n + 1) * T, f"{where}: decode cache holds {n_tok} rows"
                assert np.array_equal(ck, host[l]["k"]), f"{where}: decode cache K rows differ"
                assert np.array_equal(cv, host[l]["v"]), f"{where}: decode cache V rows differ"
                summary["near_tie_diffs"] += rep["near_tie_diffs"]
                summary["straddle_oracle"] += rep["straddle_oracle"]
                summary["straddle_gpu"] += rep["straddle_gpu"]
                for g, gap in rep["diverged_heads"]:
                    summary["divergences"].append({"frame": n, "layer": l, "kv_head": g, "gap": gap})
                    if summary["first_divergence"] is None:
                        summary["first_divergence"] = n
                for key in ("o_max", "o_mean", "score_rel_max"):
                    summary[key] = max(summary[key], rep[key])
                before[l] = gpu_state_as_oracle(after, wl.dtype)
    finally:
        pool.shutdown()
        stepper.close()
    summary["max_divergence_gap"] = max((d["gap"] for d in summary["divergences"]), default=None)
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
