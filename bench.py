"""Benchmark of the StateKV per-frame video-prefill step on one MI355X.

A step is one frame of the video through every layer of the stack (attention
with fused importance scoring, Top-B selection, state update, decode-cache
append), in one skv_frame_step call.  The whole 512-frame video's Q/K/V are
generated on the device and resident in HBM before timing; after the last
frame the stream restarts from frame 0 with an empty state (skv_reset).

Reported: frames/s over the K timed frames (host wall clock between two
device synchronisations), per-stage kernel times from HIP events recorded on
the library's stream, the attention kernel's roofline position, per-frame
latency against frame index, and the fp64 CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "video-prefill frames/s (7B shape, 512 frames); % bf16 MFMA peak; HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
ATTN_SOURCES = ["paper_2605_31598_amd/csrc/attn_mfma.hip", "paper_2605_31598_amd/csrc/internal.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_mfma_vlm7b_28layer_traffic.txt")


def attn_source_hash():
    """Hash of what the attention kernel is built from: its source file and the
    launch-argument struct it reads (the rest of internal.h serves other kernels)."""
    h = hashlib.sha256()
    with open(os.path.join(ROOT, ATTN_SOURCES[0]), "rb") as f:
        h.update(f.read())
    with open(os.path.join(ROOT, ATTN_SOURCES[1]), "r") as f:
        text = f.read()
    start = text.index("struct AttnArgs {")
    h.update(text[start:text.index("};", start) + 2].encode())
    return h.hexdigest()[:16]


def stored_traffic():
    """HBM bytes per attention launch from the committed rocprofv3 counter summary,
    valid only while the attention source is unchanged since the counters were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line:
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("attn_source_sha256_16") != attn_source_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def attention_flops(wl, S):
    """Causal-exact algorithmic FLOPs of one frame over all layers: QK^T and PV once."""
    T = wl.tokens_per_frame
    return 4 * wl.head_dim * wl.n_q_heads * (T * S + T * (T + 1) // 2) * wl.n_layers


def executed_mfma_flops(wl, S):
    """MFMA FLOPs the attention kernel issues: K Q^T in both sweeps plus P V once, over
    whole 32-row wave blocks and 128-key tiles."""
    T = wl.tokens_per_frame
    rows = -(-(wl.group * T) // 32) * 32
    keys = -(-(S + T) // 128) * 128
    return 3 * 2 * rows * keys * wl.head_dim * wl.n_kv_heads * wl.n_layers


def refresh_bytes(wl, S, n_qtiles, admitted):
    """Algorithmic HBM bytes of one refresh launch: score finalisation and selection
    (column-sum partials and state positions read; pool scores/positions, retained
    scores and admit lists written), the admitted rows' K/V copied into the state
    (read + write, plus position and score), and the frame's K/V appended to the
    decode cache (read + write).  `admitted` = mean admitted rows per (layer, KV head)."""
    LH = wl.n_layers * wl.n_kv_heads
    T, rb = wl.tokens_per_frame, wl.head_dim * 2
    P = S + T
    select = LH * (n_qtiles * P * 4 + S * 4 + P * 8 + 2 * T * 4 + S * 4)
    update = LH * admitted * (2 * 2 * rb + 8)
    append = LH * T * rb * 2 * 2
    return select + update + append


def full_attention_flops(wl, n):
    """Causal-exact FLOPs of frame n under streaming full attention (all n*T earlier tokens)."""
    return attention_flops(wl, n * wl.tokens_per_frame)


def baselines(wl, q_all, k_all, v_all, out, stream, statekv_ms):
    """The paper's two comparison systems on the same resident inputs, outside the timed
    region of the main line: streaming full attention over the decode cache (one whole
    video, per-frame times) and the recency window of B tokens (one video); and StateKV
    with YaRN-scaled RoPE applied inside the step at virtual positions (one video)."""
    from paper_2605_31598_amd import FrameStepper
    import torch

    N, T = wl.n_frames, wl.tokens_per_frame
    res = {}
    runs = {"full": dict(policy="full"), "recent": dict(policy="recent"),
            "statekv_yarn": dict(policy="statekv", rope="yarn", rope_theta=1e6, rope_factor=4.0, rope_orig_max=32768)}
    for name, kw in runs.items():
        policy = kw["policy"]
        st = FrameStepper.from_workload(wl, stream=stream, **kw)
        try:
            for f in range(4):  # warm the kernels, then restart the stream
                st.step(q_all[f], k_all[f], v_all[f], out)
            st.reset()
            torch.cuda.synchronize()
            st.timing_start(N)
            t0 = time.perf_counter()
            for f in range(N):
                st.step(q_all[f], k_all[f], v_all[f], out)
            torch.cuda.synchronize()
            wall = time.perf_counter() - t0
            ms = st.timing_stop(N).astype(np.float64)
        finally:
            st.close()
        frame_ms = ms.sum(axis=1)
        entry = {"frames_per_s": round(N / wall, 2), "video_s": round(wall, 3),
                 "frame_ms_at": {str(f): round(float(frame_ms[f]), 4) for f in (0, 11, 64, 128, 256, N - 1) if f < N}}
        if policy == "full":
            alg = np.array([full_attention_flops(wl, f) for f in range(N)], dtype=np.float64)
            last = slice(N - 64, N)
            entry["attention_tflops_last_64_frames"] = round(float(alg[last].sum() / (ms[last, 0].sum() * 1e-3) / 1e12), 1)
            entry["attention_frac_of_bf16_peak_last_64"] = round(float(alg[last].sum() / (ms[last, 0].sum() * 1e-3) / 1e12)
                                                                 / PEAK_BF16_TFLOPS, 4)
            slower = np.nonzero(frame_ms > statekv_ms)[0]
            entry["crossover_frame"] = int(slower[0]) if slower.size else None
            entry["statekv_speedup_at_last_frame"] = round(float(frame_ms[-1] / statekv_ms), 2)
        res[name] = entry
        print(f"[bench] {name}: {entry['frames_per_s']} frames/s over one video", file=sys.stderr, flush=True)
    res["statekv_frame_ms_state_full"] = round(statekv_ms, 4)
    return res


def diagnostics_bench(stream, n_frames=32, budgets=(16, 256, 1024)):
    """The appendix's assumption diagnostics on a synthetic stream of the one-layer 7B shape,
    keeping every token so each frame's scores cover its whole history.  On i.i.d. inputs
    they describe the generator, not a video model: reported for completeness."""
    from paper_2605_31598_amd import FrameStepper
    from paper_2605_31598_amd import diagnostics as dg
    from workloads import CONFIGS
    from workloads import device as wdev
    from workloads import generate as gen
    import torch

    wl = CONFIGS["vlm7b_1layer"]
    wl = wl.with_(capacity=n_frames * wl.tokens_per_frame, n_frames=n_frames)
    T, d = wl.tokens_per_frame, wl.head_dim
    st = FrameStepper.from_workload(wl, stream=stream)
    q = torch.empty((n_frames, 1, wl.n_q_heads, T, d), dtype=torch.bfloat16, device="cuda")
    k = torch.empty((n_frames, 1, wl.n_kv_heads, T, d), dtype=torch.bfloat16, device="cuda")
    v = torch.empty_like(k)
    for t, tid in ((q, gen.TENSOR_Q), (k, gen.TENSOR_K), (v, gen.TENSOR_V)):
        wdev.fill_iid(t, [gen.stream_key(wl.seed, 0, f, tid) for f in range(n_frames)], "bf16")
    out = torch.empty((1, wl.n_q_heads, T, d), dtype=torch.bfloat16, device="cuda")
    frames = []
    try:
        for n in range(n_frames):
            st.step(q[n], k[n], v[n], out)
            s, p = dg.layer_frames_from_stepper(st, 0, T)
            frames.append((s, p, wl.pos_offset + n * T))
    finally:
        st.close()
    res = dg.summarise(frames, list(budgets))
    return {"stream": f"{wl.name}, {n_frames} frames, i.i.d. inputs", **{str(b): {k2: round(v2, 4) for k2, v2 in r.items()}
                                                                       for b, r in res.items()}}


def decode_bench(wl, q_all, k_all, v_all, out, stream, n_calls=32):
    """Decoding after a whole video: one token per call over the detailed cache D of every
    layer (all T * N video tokens), the step the paper runs after prefill.  HBM-bound: each
    call reads all of D's K and V once."""
    from paper_2605_31598_amd import FrameStepper
    import torch

    N, T, L = wl.n_frames, wl.tokens_per_frame, wl.n_layers
    st = FrameStepper.from_workload(wl, stream=stream, max_decode_tokens=n_calls + 8)
    try:
        for f in range(N):
            st.step(q_all[f], k_all[f], v_all[f], out)
        g = torch.Generator(device="cuda").manual_seed(wl.seed + 1)
        q = torch.randn((n_calls + 8, L, wl.n_q_heads, 1, wl.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        k = torch.randn((n_calls + 8, L, wl.n_kv_heads, 1, wl.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        v = torch.randn((n_calls + 8, L, wl.n_kv_heads, 1, wl.head_dim), generator=g, device="cuda").to(torch.bfloat16)
        o = torch.empty((L, wl.n_q_heads, 1, wl.head_dim), dtype=torch.bfloat16, device="cuda")
        for i in range(8):  # warm-up calls
            st.decode(q[i], k[i], v[i], o)
        torch.cuda.synchronize()
        st.timing_start(n_calls)
        t0 = time.perf_counter()
        for i in range(8, 8 + n_calls):
            st.decode(q[i], k[i], v[i], o)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = st.timing_stop(n_calls).astype(np.float64)
    finally:
        st.close()
    keys = N * T + 8 + np.arange(n_calls) + 1  # keys per query of each timed call
    kv_bytes = keys * L * wl.n_kv_heads * wl.head_dim * 2 * 2  # K and V of every key, read once
    att = ms[:, 0]
    gbs = float(kv_bytes.sum() / (att.sum() * 1e-3) / 1e9)
    return {"kernel": "decode_split_kernel<128> + decode_combine_kernel<128>", "tokens_per_call": 1,
            "cached_tokens_per_kv_head": int(N * T), "calls": n_calls,
            "ms_per_call": round(float(att.mean()), 4), "tokens_per_s": round(n_calls / wall, 1),
            "kv_bytes_per_call": float(kv_bytes.mean()), "GBps": round(gbs, 1), "peak_GBps": PEAK_HBM_GBS,
            "frac": round(gbs / PEAK_HBM_GBS, 4), "append_ms_per_call": round(float(ms[:, 1].mean()), 4)}


def per_layer_bench(wl, q_all, k_all, v_all, out, stream, n_frames=16):
    """The real-model calling pattern: one skv_frame_step per layer (a model interleaves its
    projections and MLP between them), timed at state full.  A one-layer call is too small to
    fill the device, so its attention splits the keys (statistics, output shares, and their sum
    in the refresh launch)."""
    from paper_2605_31598_amd import FrameStepper
    import torch

    L, first = wl.n_layers, wl.full_from_frame + 4
    st = FrameStepper.from_workload(wl, stream=stream)

    def frames(f0):
        for f in range(f0, f0 + n_frames):
            for l in range(L):
                st.step(q_all[f][l:l + 1], k_all[f][l:l + 1], v_all[f][l:l + 1], out[l:l + 1],
                        layer_begin=l, layer_count=1)

    try:
        for f in range(first):
            st.step(q_all[f], k_all[f], v_all[f], out)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        frames(first)  # wall clock, no events
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        st.timing_start(n_frames * L)  # then the same number of frames with per-call events
        frames(first + n_frames)
        ms = st.timing_stop(n_frames * L).astype(np.float64)
    finally:
        st.close()
    return {"layers_per_call": 1, "timed_frames_at_state_full": n_frames, "frames_per_s": round(n_frames / wall, 2),
            "ms_per_frame": round(1e3 * wall / n_frames, 4),
            "attention_ms_per_call": round(float(ms[:, 0].mean()), 4),
            "refresh_ms_per_call": round(float(ms[:, 1].mean()), 4)}


def large_bench(stream, name="vlm72b_80layer", timed=16, kv_heads=None):
    """The 72B-shaped stack (80 layers, 64 Q / 8 KV heads, 256 tokens/frame, capacity 4096,
    low-rank keys built on the device): the first frames fill the state, then `timed`
    frames run at state full, all 80 layers per call.  Reported beside the 7B line.
    kv_heads < 8 runs one GPU's share of a head-sharded stack (kv_heads KV heads and
    their query heads on each GPU; the heads need nothing from each other)."""
    from paper_2605_31598_amd import FrameStepper
    from workloads import CONFIGS
    from workloads import device as wdev
    from workloads import generate as gen
    import torch

    wl = CONFIGS[name]
    if kv_heads is not None:
        wl = wl.with_(n_kv_heads=kv_heads, n_q_heads=wl.group * kv_heads)
    L, Hq, Hkv, T, d = wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.tokens_per_frame, wl.head_dim
    fill = -(-wl.capacity // T)  # frames until the state is full
    F = fill + timed
    q = torch.empty((F, L, Hq, T, d), dtype=torch.bfloat16, device="cuda")
    k = torch.empty((F, L, Hkv, T, d), dtype=torch.bfloat16, device="cuda")
    v = torch.empty_like(k)
    for t, tid in ((q, gen.TENSOR_Q), (v, gen.TENSOR_V)):
        wdev.fill_iid(t, [gen.stream_key(wl.seed, l, f, tid) for f in range(F) for l in range(L)], "bf16")
    kl = torch.empty((F, Hkv, T, d), dtype=torch.bfloat16, device="cuda")
    for l in range(L):
        wdev.fill_lowrank_keys(kl, wl, l, range(F))
        k[:, l].copy_(kl)
    del kl
    out = torch.empty((L, Hq, T, d), dtype=torch.bfloat16, device="cuda")
    st = FrameStepper.from_workload(wl, max_frames=F, stream=stream)
    try:
        for n in range(fill):
            st.step(q[n], k[n], v[n], out)
        torch.cuda.synchronize()
        st.timing_start(timed)
        t0 = time.perf_counter()
        for n in range(fill, F):
            st.step(q[n], k[n], v[n], out)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        stages = st.timing_stop(timed).astype(np.float64)
    finally:
        st.close()
    del q, k, v
    att = stages[:, 0]
    alg = attention_flops(wl, wl.capacity)
    exe = executed_mfma_flops(wl, wl.capacity)
    frame_ms = stages.sum(axis=1)
    shards = CONFIGS[name].n_kv_heads // wl.n_kv_heads
    res = {"workload": name if shards == 1 else f"{name}, one GPU's share of {shards}-way KV-head sharding",
           "layers": L, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d, "tokens_per_frame": T,
           "capacity": wl.capacity, "inputs": "i.i.d. N(0,1) Q and V, low-rank keys (rank 16 + noise), bf16",
           "timed_frames_at_state_full": timed, "frames_per_s": round(timed / wall, 2),
           "ms_per_frame": round(1e3 * wall / timed, 4), "attention_ms": round(float(att.mean()), 4),
           "refresh_ms": round(float(stages[:, 1].mean()), 4),
           "attention_tflops": round(alg / (att.mean() * 1e-3) / 1e12, 1),
           "attention_frac_of_bf16_peak": round(alg / (att.mean() * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "executed_mfma_frac": round(exe / (att.mean() * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "flatness_max_dev": round(float(np.max(np.abs(frame_ms / np.median(frame_ms) - 1.0))), 4)}
    print(f"[bench] {name}: {res['frames_per_s']} frames/s at state full", file=sys.stderr, flush=True)
    return res


def copy_bandwidth(n_bytes=1 << 30, reps=5):
    """Read + write GB/s of the runtime's device-to-device copy of 1 GiB: the practical
    streaming rate the refresh launch's GB/s is set against."""
    import torch

    src = torch.ones(n_bytes // 2, dtype=torch.int16, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    b.synchronize()
    gbs = 2 * n_bytes * reps / (a.elapsed_time(b) * 1e-3) / 1e9
    del src, dst
    return round(gbs, 1)


def cpu_baseline(wl, seconds):
    """The fp64 oracle on a bounded sample: layer 0, frames from state-full onward, on a
    full state of the most recent tokens; scaled to frames/s of the whole stack."""
    from oracle import statekv_oracle as orc
    from workloads import generate as gen

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    n0 = wl.full_from_frame + 1
    # state: most recent B tokens entering frame n0
    S = wl.state_size(n0)
    ks, vs, ps = [], [], []
    for f in range(max(0, n0 - (-(-S // wl.tokens_per_frame))), n0):
        x = gen.frame_inputs(wl, 0, f)
        ks.append(gen.to_f64(x["k"], wl.dtype))
        vs.append(gen.to_f64(x["v"], wl.dtype))
        ps.append(orc.frame_positions(f, wl.tokens_per_frame, wl.pos_offset))
    H = wl.n_kv_heads
    st = orc.LayerState(np.tile(np.concatenate(ps)[-S:], (H, 1)), np.concatenate(ks, axis=1)[:, -S:],
                        np.concatenate(vs, axis=1)[:, -S:], np.zeros((H, S)))
    times = []
    t_start = time.perf_counter()
    n = n0
    while time.perf_counter() - t_start < seconds and n < wl.n_frames:
        x = gen.frame_inputs_f64(wl, 0, n)
        t0 = time.perf_counter()
        r = orc.frame_step(st, x["q"], x["k"], x["v"], n, wl.capacity, wl.scale, wl.pos_offset)
        times.append(time.perf_counter() - t0)
        st = r.state
        n += 1
    per_layer_frame = float(np.mean(times))
    return {
        "value": 1.0 / (per_layer_frame * wl.n_layers),
        "unit": "frames/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"fp64 numpy oracle, layer 0 of {wl.n_layers}, frames {n0}..{n - 1} on a full state "
                  f"({len(times)} layer-frames, {per_layer_frame * 1e3:.1f} ms each; input generation excluded); "
                  f"scaled by {wl.n_layers} layers",
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1536, help="timed frames (the video restarts after its last frame)")
    ap.add_argument("--warmup", type=int, default=512, help="untimed frames before timing")
    ap.add_argument("--workload", default="vlm7b_28layer")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-baselines", action="store_true",
                    help="skip the runs reported beside the main line (Full SA, recency window, YaRN, decode, "
                         "diagnostics, the 72B-shaped stack)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (the step shards by KV head "
              "and by layer with no exchange; see the design notes). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2605_31598_amd import FrameStepper
    from workloads import CONFIGS
    from workloads import device as wdev
    from workloads import generate as gen

    if args.copy_calibration:
        src = torch.ones(1 << 29, dtype=torch.int16, device="cuda")  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": src.numel() * 2, "copy_calibration_bytes_written": src.numel() * 2,
                          "launches": 3}))
        return

    wl = CONFIGS[args.workload]
    if wl.dtype != "bf16":
        raise SystemExit("the benchmark runs bf16 workloads")
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    L, N, Hq, Hkv, T, d = wl.n_layers, wl.n_frames, wl.n_q_heads, wl.n_kv_heads, wl.tokens_per_frame, wl.head_dim

    # whole video resident in HBM, generated on the device (untimed)
    q_all = torch.empty((N, L, Hq, T, d), dtype=torch.bfloat16, device="cuda")
    k_all = torch.empty((N, L, Hkv, T, d), dtype=torch.bfloat16, device="cuda")
    v_all = torch.empty((N, L, Hkv, T, d), dtype=torch.bfloat16, device="cuda")
    for t, tid in ((q_all, gen.TENSOR_Q), (k_all, gen.TENSOR_K), (v_all, gen.TENSOR_V)):
        keys = [gen.stream_key(wl.seed, l, f, tid) for f in range(N) for l in range(L)]
        wdev.fill_iid(t, keys, "bf16")
    out = torch.empty((L, Hq, T, d), dtype=torch.bfloat16, device="cuda")
    print(f"[bench] {wl.name}: inputs resident ({(q_all.numel() + k_all.numel() + v_all.numel()) * 2 / 1e9:.1f} GB)",
          file=sys.stderr, flush=True)

    st = FrameStepper.from_workload(wl, stream=stream)
    counter = {"i": 0}

    def run(n_frames):
        for _ in range(n_frames):
            f = counter["i"] % N
            if f == 0 and counter["i"] > 0:
                st.reset()
            st.step(q_all[f], k_all[f], v_all[f], out)
            counter["i"] += 1

    run(args.warmup)
    torch.cuda.synchronize()
    first_frame = counter["i"] % N
    st.timing_start(args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(args.steps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    stages = st.timing_stop(args.steps)  # [K, 2] ms: attention, refresh
    # rows admitted by the last timed frame (its positions are the newest in the state)
    last_pos0 = wl.pos_offset + ((counter["i"] - 1) % N) * T
    admitted = float(np.mean([(st.read_state(l)["pos"] >= last_pos0).sum(axis=1).mean() for l in range(L)]))
    st.close()
    elapsed = t1 - t0
    fps = args.steps / elapsed
    print(f"[bench] timed {args.steps} frames in {elapsed:.3f} s", file=sys.stderr, flush=True)

    frames = (first_frame + np.arange(args.steps)) % N
    S = np.minimum(wl.capacity, frames * T)
    attn_ms = stages[:, 0].astype(np.float64)
    alg = np.array([attention_flops(wl, int(s)) for s in S], dtype=np.float64)
    exe = np.array([executed_mfma_flops(wl, int(s)) for s in S], dtype=np.float64)
    achieved = alg.sum() / (attn_ms.sum() * 1e-3) / 1e12
    executed = exe.sum() / (attn_ms.sum() * 1e-3) / 1e12
    n_qtiles = -(-(wl.group * T) // 256)
    ref_b = np.array([refresh_bytes(wl, int(s), n_qtiles, admitted) for s in S], dtype=np.float64)
    refresh_gbs = float(ref_b.sum() / (stages[:, 1].astype(np.float64).sum() * 1e-3) / 1e9)

    frame_ms = stages.sum(axis=1)
    full = frames >= wl.full_from_frame
    per_index = {}
    for f, ms in zip(frames[full], frame_ms[full]):
        per_index.setdefault(int(f), []).append(float(ms))
    med_by_frame = np.array([np.median(v) for _, v in sorted(per_index.items())]) if per_index else np.array([0.0])
    med = float(np.median(med_by_frame))
    traffic = stored_traffic()

    result = {
        "metric": METRIC,
        "value": round(fps, 3),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": L, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d,
                   "tokens_per_frame": T, "frames_per_video": N, "capacity": wl.capacity,
                   "layers_per_call": L, "inputs": "i.i.d. N(0,1) bf16, generated in HBM"},
        "roofline": {
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "kernel": "attn_mfma_kernel<128>",
            "flops_per_launch": float(alg.mean()),
            "avg_launch_ms": float(attn_ms.mean()),
            "executed_mfma_tflops": round(executed, 2),
            "executed_frac": round(executed / PEAK_BF16_TFLOPS, 4),
        },
        "stages_ms_mean": {n: float(stages[:, i].mean()) for i, n in enumerate(("attention", "refresh"))},
        "hbm": {
            "kernel": "refresh_kernel (selection + state update + decode-cache append)",
            "bytes_per_launch": float(ref_b.mean()),
            "admitted_rows_per_head": round(admitted, 1),
            "GBps": round(refresh_gbs, 1),
            "peak_GBps": PEAK_HBM_GBS,
            "frac": round(refresh_gbs / PEAK_HBM_GBS, 4),
        },
        "latency": {
            "frame_ms_median_state_full": round(med, 4),
            "flatness_max_dev": round(float(np.max(np.abs(med_by_frame / med - 1.0))), 4) if med > 0 else None,
            "frame_ms_first_frames": [round(float(x), 4) for x in frame_ms[:min(16, len(frame_ms))]],
            "from_frame": int(wl.full_from_frame),
        },
    }
    if not args.no_baselines:
        result["baselines"] = baselines(wl, q_all, k_all, v_all, out, stream, med)
        result["decode"] = decode_bench(wl, q_all, k_all, v_all, out, stream)
        result["per_layer"] = per_layer_bench(wl, q_all, k_all, v_all, out, stream)
        result["diagnostics"] = diagnostics_bench(stream)
        result["vlm72b"] = large_bench(stream)
        result["vlm72b_shard8"] = large_bench(stream, kv_heads=1)
        result["hbm"]["copy_GBps"] = copy_bandwidth()
        result["hbm"]["frac_of_copy"] = round(result["hbm"]["GBps"] / result["hbm"]["copy_GBps"], 4)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
