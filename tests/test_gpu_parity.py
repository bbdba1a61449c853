"""GPU parity of skv_frame_step against the fp64 oracle (through the C ABI).

Run on an MI355X: python -u -m pytest tests -m gpu -x -v --timeout 120 --timeout-method thread
"""
from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import statekv_oracle as orc  # noqa: E402
from paper_2605_31598_amd import FrameStepper, StateKVError  # noqa: E402
from workloads import CONFIGS, WorkloadConfig  # noqa: E402
from workloads import generate as gen  # noqa: E402

from .gpu_harness import (  # noqa: E402
    NEAR_TIE_REL, compare_step, frame_tensors, gpu_state_as_oracle, oracle_step, recent_state, run_tracking, say,
    to_device,
)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


# --------------------------------------------------------------------------
# whole videos, end to end: the GPU's state evolves by itself from the empty
# state; every frame is checked against the oracle, and every frame where the
# GPU keeps another set than the oracle's own evolution must be a near-tie
# --------------------------------------------------------------------------
def _assert_divergences_at_near_ties(s):
    assert len(s["divergences"]) == s["near_tie_diffs"]
    for d in s["divergences"]:
        assert d["gap"] <= NEAR_TIE_REL, f"divergence away from a near-tie: {d}"


def test_tiny_f32_whole_video():
    wl = CONFIGS["tiny_f32"]
    s = run_tracking(wl, wl.n_frames, [0])
    say(f"tiny_f32: {s}")
    assert s["first_divergence"] is None
    assert s["o_max"] <= 1e-5


def test_vlm7b_1layer_whole_video():
    wl = CONFIGS["vlm7b_1layer"]
    s = run_tracking(wl, wl.n_frames, [0], log_every=8)
    say(f"vlm7b_1layer: {s}")
    _assert_divergences_at_near_ties(s)


def test_vlm7b_28layer_whole_video():
    """All 512 frames of the 7B stack, all 28 layers per call as the benchmark runs
    them; layers 0 and 27 checked every frame (the others get zero inputs)."""
    wl = CONFIGS["vlm7b_28layer"]
    s = run_tracking(wl, wl.n_frames, [0, 27], log_every=32)
    _assert_divergences_at_near_ties(s)
    s["divergences"] = s["divergences"][:8]
    say(f"vlm7b_28layer whole video: {s}")


def test_vlm72b_80layer_stream_past_state_full():
    """The 72B stack from the empty state through 64 frames past state-full (frame 16),
    all 80 layers per call; layers 0 and 79 checked every frame."""
    wl = CONFIGS["vlm72b_80layer"]
    n = wl.full_from_frame + 64
    s = run_tracking(wl, n, [0, 79], log_every=8)
    say(f"vlm72b_80layer frames 0..{n - 1}: {s}")
    _assert_divergences_at_near_ties(s)


def test_stress_stream_past_state_full():
    """The stress layer (duplicate and heavy keys) from the empty state through 64 frames
    past state-full (frame 12)."""
    wl = CONFIGS["stress_1layer"]
    n = wl.full_from_frame + 64
    s = run_tracking(wl, n, [0], log_every=8)
    say(f"stress_1layer frames 0..{n - 1}: {s}")
    _assert_divergences_at_near_ties(s)
    # exact ties of the oracle (duplicate keys) are exact on the GPU too, and go the same way
    assert all(d["gap"] > 0.0 for d in s["divergences"]), s["divergences"]
    assert s["straddle_gpu"] == s["straddle_oracle"] > 0


# --------------------------------------------------------------------------
# edge shapes: ragged rows and keys, G = 1, B = 0, B < T, T = 1, pool never full
# --------------------------------------------------------------------------
EDGE = [
    # name, H_q, H_kv, d, T, B, N, dtype
    ("ragged_T37_G1", 4, 4, 128, 37, 50, 5, "bf16"),
    ("capacity0", 8, 2, 64, 5, 0, 4, "bf16"),
    ("B_lt_T", 8, 2, 128, 20, 7, 5, "bf16"),
    ("T1", 4, 1, 128, 1, 3, 6, "bf16"),
    ("never_prunes", 6, 2, 128, 100, 1000, 4, "bf16"),
    ("f32_d64", 4, 2, 64, 16, 32, 5, "f32"),
    ("f32_d128_ragged", 4, 2, 128, 33, 40, 5, "f32"),
    ("bf16_d64_multi_tile", 16, 2, 64, 300, 600, 4, "bf16"),
    ("bf16_G7_T196_B300", 28, 4, 128, 196, 300, 4, "bf16"),
    # frames over 1024 tokens: the refresh keeps its admit lists in global memory
    ("T1100_global_admit_lists", 2, 1, 64, 1100, 1500, 3, "bf16"),
]


@pytest.mark.parametrize("name,Hq,Hkv,d,T,B,N,dtype", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes(name, Hq, Hkv, d, T, B, N, dtype):
    wl = WorkloadConfig(name, 1, Hq, Hkv, d, T, N, B, dtype, "iid", 777 + len(name), pos_offset=13)
    s = run_tracking(wl, N, [0])
    say(f"{name}: {s}")


def test_two_layer_stack_layer_by_layer_calls():
    """Real-model calling pattern: one call per layer, in order."""
    wl = WorkloadConfig("two_layer", 2, 8, 2, 128, 24, 4, 40, "bf16", "iid", 4242)
    st = FrameStepper.from_workload(wl)
    own = {l: orc.LayerState.empty(2, 128) for l in range(2)}
    try:
        out = torch.empty((1, 8, 24, 128), dtype=torch.bfloat16, device="cuda")
        for n in range(wl.n_frames):
            for l in range(2):
                x = gen.frame_inputs(wl, l, n)
                st.step(to_device(x["q"][None], "bf16"), to_device(x["k"][None], "bf16"),
                        to_device(x["v"][None], "bf16"), out, layer_begin=l, layer_count=1)
                res = oracle_step(wl, own[l], x, n)
                after = st.read_state(l)
                compare_step(res, out[0].float().cpu().numpy().astype(np.float64), after["pool_score"],
                             after["pool_pos"], after["pos"], wl.capacity, "bf16", f"layer {l} frame {n}")
                own[l] = gpu_state_as_oracle(after, "bf16")
    finally:
        st.close()


# --------------------------------------------------------------------------
# full sizes, in the launch configuration the benchmark times (all layers per call)
# --------------------------------------------------------------------------
FULL = [("vlm7b_28layer", [0, 13, 27], 40), ("vlm72b_80layer", [0, 79], 20), ("stress_1layer", [0], 30)]


@pytest.mark.parametrize("name,layers,frame", FULL, ids=[f[0] for f in FULL])
def test_full_size_one_frame_on_forced_full_state(name, layers, frame):
    wl = CONFIGS[name]
    forced = {l: recent_state(wl, l, frame) for l in layers}
    s = run_tracking(wl, 1, layers, start_frame=frame, forced=forced)
    say(f"{name} frame {frame}: {s}")
    if name == "stress_1layer":
        # duplicate keys tie exactly across the capacity boundary: the tie pass decides
        assert s["straddle_oracle"] >= 1 and s["straddle_gpu"] >= 1


PER_LAYER = [("vlm7b_28layer", [0, 27], 40), ("vlm72b_80layer", [0, 79], 20)]


@pytest.mark.parametrize("name,layers,frame", PER_LAYER, ids=[f[0] for f in PER_LAYER])
def test_full_size_one_layer_per_call_on_forced_full_state(name, layers, frame):
    """Real-model calling pattern at full size: one call per layer, each too small to
    fill the device, so the attention splits the keys over 10 (7B) or 4 (72B) ranges."""
    wl = CONFIGS[name]
    forced = {l: recent_state(wl, l, frame) for l in layers}
    s = run_tracking(wl, 2, layers, start_frame=frame, forced=forced, per_layer=True)
    say(f"{name} frames {frame}-{frame + 1}, one layer per call: {s}")


T259 = CONFIGS["vlm7b_28layer"].with_(name="vlm7b_28layer_t259", tokens_per_frame=259)


@pytest.mark.parametrize("per_layer", [False, True], ids=["whole_stack", "one_layer_per_call"])
def test_259_tokens_per_frame_on_forced_full_state(per_layer):
    """The 7B-shaped stack at 259 tokens per frame (the paper's InternVL3 setting): 1813
    query rows per KV head, not a multiple of the 32-row wave blocks.  One layer per call
    splits the keys 8 ways (256 workgroups, as many as the device has compute units)."""
    wl, frame = T259, 12
    layers = [0, 27]
    forced = {l: recent_state(wl, l, frame) for l in layers}
    s = run_tracking(wl, 2, layers, start_frame=frame, forced=forced, per_layer=per_layer)
    say(f"{wl.name} frames {frame}-{frame + 1}{', one layer per call' if per_layer else ''}: {s}")


def test_stress_ties_resolved_by_position():
    """Stress keys on the most recent state entering frame 15: exact duplicate rows give
    bit-equal scores on both sides, and in at least one KV head the tied entries straddle
    the capacity boundary (kv head 7: 26 tied scores for 14 places), so the lowest
    positions must win."""
    wl = CONFIGS["stress_1layer"].with_(n_frames=16)
    s = run_tracking(wl, 1, [0], start_frame=15, forced={0: recent_state(wl, 0, 15)})
    say(f"stress frame 15: {s}")
    assert s["straddle_oracle"] >= 1, "the oracle's pool has no tie across the boundary"
    assert s["straddle_gpu"] >= 1, "the GPU's pool has no tie across the boundary"


@pytest.mark.parametrize("Hq,Hkv,d,T,B,N", [(8, 2, 128, 40, 100, 6), (28, 4, 128, 196, 2048, 13)],
                         ids=["small", "vlm7b_layer"])
def test_zero_queries_keep_the_earliest_tokens(Hq, Hkv, d, T, B, N):
    """Q = 0: attention is uniform, every state key and frame token 0 tie exactly (on
    the GPU too: equal logits give equal exponentials summed in the same order), so
    once the state is full B + 1 entries tie for B places and the tie rule keeps the
    earliest B tokens forever (closed form of the selection)."""
    wl = WorkloadConfig("zero_q", 1, Hq, Hkv, d, T, N, B, "bf16", "iid", 5150, pos_offset=7)
    st = FrameStepper.from_workload(wl)
    own = orc.LayerState.empty(Hkv, d)
    straddle = 0
    try:
        out = torch.empty((1, Hq, T, d), dtype=torch.bfloat16, device="cuda")
        for n in range(N):
            x = gen.frame_inputs(wl, 0, n)
            x["q"] = np.zeros_like(x["q"])
            st.step(to_device(x["q"][None], "bf16"), to_device(x["k"][None], "bf16"),
                    to_device(x["v"][None], "bf16"), out)
            res = oracle_step(wl, own, x, n)
            after = st.read_state(0)
            rep = compare_step(res, out[0].float().cpu().numpy().astype(np.float64), after["pool_score"],
                               after["pool_pos"], after["pos"], B, "bf16", f"zero_q frame {n}")
            assert rep["near_tie_diffs"] == 0
            seen = (n + 1) * T
            earliest = wl.pos_offset + np.arange(min(B, seen))
            for g in range(Hkv):
                assert np.array_equal(np.sort(after["pos"][g]), earliest), f"frame {n} kv head {g}"
            if n >= wl.full_from_frame:
                assert rep["straddle_gpu"] == Hkv and rep["straddle_oracle"] == Hkv, rep
            straddle += rep["straddle_gpu"]
            own = gpu_state_as_oracle(after, "bf16")
    finally:
        st.close()
    say(f"zero_q {Hq}/{Hkv} T={T} B={B}: straddling ties on the GPU in {straddle} head-frames")


# --------------------------------------------------------------------------
# determinism, errors, device generator
# --------------------------------------------------------------------------
def test_bitwise_deterministic():
    wl = CONFIGS["vlm7b_1layer"]
    outs = []
    for rep in range(2):
        st = FrameStepper.from_workload(wl, max_frames=8)
        out = torch.empty((1, 28, 196, 128), dtype=torch.bfloat16, device="cuda")
        res = []
        for n in range(8):
            q, k, v, _ = frame_tensors(wl, n, [0])
            st.step(q, k, v, out)
            res.append(out.clone())
        s = st.read_state(0)
        st.close()
        outs.append((torch.stack(res).cpu(), s))
    assert torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16))
    for key in ("pos", "score", "pool_score", "pool_pos", "k", "v"):
        assert np.array_equal(outs[0][1][key], outs[1][1][key]), key


def test_error_statuses_on_device():
    wl = WorkloadConfig("err", 2, 4, 2, 64, 8, 2, 8, "bf16", "iid", 1)
    st = FrameStepper.from_workload(wl)
    try:
        q, k, v, _ = frame_tensors(wl, 0, [0, 1])
        out = torch.empty((2, 4, 8, 64), dtype=torch.bfloat16, device="cuda")
        with pytest.raises(StateKVError, match="SKV_ERR_ORDER"):
            st.step(q[1:], k[1:], v[1:], out[1:], layer_begin=1, layer_count=1)
        from paper_2605_31598_amd import binding as B
        with pytest.raises(StateKVError, match="SKV_ERR_INVALID_ARG"):
            B.skv_frame_step(st.ctx, 0, 3, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr())
        with pytest.raises(StateKVError, match="SKV_ERR_INVALID_ARG"):
            B.skv_frame_step(st.ctx, 0, 2, q.data_ptr(), 0, v.data_ptr(), out.data_ptr())
        with pytest.raises(StateKVError, match="SKV_ERR_INVALID_ARG"):  # misaligned by one bf16 element
            B.skv_frame_step(st.ctx, 0, 2, q.data_ptr() + 2, k.data_ptr(), v.data_ptr(), out.data_ptr())
        st.step(q, k, v, out)
        st.step(q, k, v, out)
        with pytest.raises(StateKVError, match="SKV_ERR_CAPACITY"):
            st.step(q, k, v, out)
        with pytest.raises(StateKVError, match="SKV_ERR_INVALID_ARG"):
            st.seek(2)
        st.reset()
        st.step(q, k, v, out)
        assert st.read_state(0)["frame"] == 1
    finally:
        st.close()


def test_device_generator_matches_host():
    from workloads import device

    wl = CONFIGS["vlm7b_28layer"]
    keys = [gen.stream_key(wl.seed, l, f, gen.TENSOR_Q) for l, f in [(0, 0), (3, 17), (27, 511)]]
    n = wl.n_q_heads * wl.tokens_per_frame * wl.head_dim
    out = torch.empty((3, n), dtype=torch.bfloat16, device="cuda")
    device.fill_iid(out, keys, "bf16")
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    for i, (l, f) in enumerate([(0, 0), (3, 17), (27, 511)]):
        assert np.array_equal(got[i], gen.frame_inputs(wl, l, f)["q"].reshape(-1))
    out32 = torch.empty((1, 2 * 16 * 64), dtype=torch.float32, device="cuda")  # V is [H_kv=2][T=16][d=64]
    t = CONFIGS["tiny_f32"]
    device.fill_iid(out32, [gen.stream_key(t.seed, 0, 5, gen.TENSOR_V)], "f32")
    assert np.array_equal(out32.cpu().numpy()[0], gen.frame_inputs(t, 0, 5)["v"].reshape(-1))


def test_device_lowrank_keys_match_host():
    """The 72B stack's low-rank keys, built on the device for the benchmark, equal the host generator's."""
    from workloads import device

    wl = CONFIGS["vlm72b_80layer"]
    frames = [0, 9, 511]
    for layer in (0, 41, 79):
        out = torch.empty((len(frames), wl.n_kv_heads, wl.tokens_per_frame, wl.head_dim), dtype=torch.bfloat16,
                          device="cuda")
        device.fill_lowrank_keys(out, wl, layer, frames)
        got = out.view(torch.int16).cpu().numpy().view(np.uint16)
        for i, f in enumerate(frames):
            assert np.array_equal(got[i], gen.frame_inputs(wl, layer, f)["k"]), (layer, f)


def test_device_stress_keys_match_host():
    """The stress layer's keys (templates and heavy rows), built on the device for the
    benchmark, equal the host generator's."""
    from workloads import device

    wl = CONFIGS["stress_1layer"]
    frames = [0, 13, 1023]
    out = torch.empty((len(frames), wl.n_kv_heads, wl.tokens_per_frame, wl.head_dim), dtype=torch.bfloat16,
                      device="cuda")
    device.fill_stress_keys(out, wl, 0, frames)
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    for i, f in enumerate(frames):
        assert np.array_equal(got[i], gen.frame_inputs(wl, 0, f)["k"]), f


SPLIT = [
    # name, layers, H_q, H_kv, d, T, B, N, policy
    ("vlm7b_1layer_key_split", 1, 28, 4, 128, 196, 1024, 8, "statekv"),
    ("two_layers_recent", 2, 8, 2, 128, 48, 100, 5, "recent"),
    ("T1100_global_lists", 1, 2, 1, 64, 1100, 1500, 3, "statekv"),
    ("capacity0", 2, 8, 2, 64, 24, 0, 3, "statekv"),
    ("full_policy", 2, 8, 2, 128, 40, 64, 4, "full"),
]


@pytest.mark.parametrize("name,L,Hq,Hkv,d,T,B,N,policy", SPLIT, ids=[x[0] for x in SPLIT])
def test_split_refresh_launches_match_the_fused_launch(name, L, Hq, Hkv, d, T, B, N, policy):
    """The refresh as three launches (selection, state update, append) gives the fused
    launch's outputs, states, pool scores and decode cache bit for bit; its stage timings
    are filled, the fused context's update and append stages read 0."""
    wl = WorkloadConfig(name, L, Hq, Hkv, d, T, N, B, "bf16", "iid", 31337, pos_offset=5)
    a = FrameStepper.from_workload(wl, policy=policy)
    b = FrameStepper.from_workload(wl, policy=policy, split_refresh=True)
    try:
        oa = torch.empty((L, Hq, T, d), dtype=torch.bfloat16, device="cuda")
        ob = torch.empty_like(oa)
        a.timing_start(N)
        b.timing_start(N)
        for n in range(N):
            q, k, v, _ = frame_tensors(wl, n, list(range(L)))
            a.step(q, k, v, oa)
            b.step(q, k, v, ob)
            assert torch.equal(oa.view(torch.int16), ob.view(torch.int16)), f"output, frame {n}"
            for l in range(L):
                sa, sb = a.read_state(l), b.read_state(l)
                for key in ("pos", "score", "k", "v", "pool_score", "pool_pos"):
                    assert np.array_equal(sa[key], sb[key]), f"{key}, layer {l} frame {n}"
        ta, tb = a.timing_stop(N), b.timing_stop(N)
        assert np.all(ta[:, 2:] == 0.0) and np.all(ta[:, 0] > 0.0)
        assert np.all(tb[:, 3] > 0.0) and np.all(tb[:, 0] > 0.0)
        if policy != "full":
            assert np.all(tb[:, 1] > 0.0) and np.all(tb[:, 2] > 0.0)
        for l in range(L):
            ca, cb = a.read_cache(l), b.read_cache(l)
            assert np.array_equal(ca[0], cb[0]) and np.array_equal(ca[1], cb[1]) and ca[2] == cb[2] == N * T
    finally:
        a.close()
        b.close()


def test_timing_stride_records_every_nth_step():
    """With a timing stride of 3, ten frame steps record events on steps 0, 3, 6 and 9
    only (four rows, each with a positive attention and refresh time); a limit of two
    recorded steps stops after steps 0 and 3; the outputs are those of an untimed context."""
    wl = WorkloadConfig("stride", 2, 8, 2, 64, 40, 10, 64, "bf16", "iid", 4242)
    L, Hq, T, d = wl.n_layers, wl.n_q_heads, wl.tokens_per_frame, wl.head_dim
    a, b, c = (FrameStepper.from_workload(wl) for _ in range(3))
    try:
        oa, ob, oc = (torch.empty((L, Hq, T, d), dtype=torch.bfloat16, device="cuda") for _ in range(3))
        a.timing_start(8, stride=3)
        b.timing_start(2, stride=3)
        for n in range(wl.n_frames):
            q, k, v, _ = frame_tensors(wl, n, list(range(L)))
            for s, o in ((a, oa), (b, ob), (c, oc)):
                s.step(q, k, v, o)
            assert torch.equal(oa.view(torch.int16), oc.view(torch.int16)), f"frame {n}"
            assert torch.equal(ob.view(torch.int16), oc.view(torch.int16)), f"frame {n}"
        ta, tb = a.timing_stop(8), b.timing_stop(8)
        assert ta.shape[0] == 4 and tb.shape[0] == 2
        assert np.all(ta[:, :2] > 0.0) and np.all(tb[:, :2] > 0.0)
    finally:
        for s in (a, b, c):
            s.close()
