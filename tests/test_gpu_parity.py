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
    compare_step, frame_tensors, gpu_state_as_oracle, oracle_step, recent_state, run_tracking, say, to_device,
)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


# --------------------------------------------------------------------------
# whole videos, every frame checked on the GPU's own state + independent run
# --------------------------------------------------------------------------
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
    s = run_tracking(wl, 1, layers, start_frame=frame, forced=forced, independent=False)
    say(f"{name} frame {frame}: {s}")


PER_LAYER = [("vlm7b_28layer", [0, 27], 40), ("vlm72b_80layer", [0, 79], 20)]


@pytest.mark.parametrize("name,layers,frame", PER_LAYER, ids=[f[0] for f in PER_LAYER])
def test_full_size_one_layer_per_call_on_forced_full_state(name, layers, frame):
    """Real-model calling pattern at full size: one call per layer, each too small to
    fill the device, so the attention splits the keys over 10 (7B) or 4 (72B) ranges."""
    wl = CONFIGS[name]
    forced = {l: recent_state(wl, l, frame) for l in layers}
    s = run_tracking(wl, 2, layers, start_frame=frame, forced=forced, independent=False, per_layer=True)
    say(f"{name} frames {frame}-{frame + 1}, one layer per call: {s}")


def test_vlm7b_28layer_stream_through_state_full():
    """First 14 frames of the 28-layer stack (state full from frame 11), layers 0 and 27 checked."""
    wl = CONFIGS["vlm7b_28layer"]
    s = run_tracking(wl, 14, [0, 27], log_every=2)
    say(f"vlm7b_28layer 14 frames: {s}")


def test_stress_ties_resolved_by_position():
    """Stress keys: exact duplicate rows inside the state give bit-equal GPU scores; the lower position wins."""
    wl = CONFIGS["stress_1layer"].with_(n_frames=16)
    s = run_tracking(wl, 2, [0], start_frame=14, forced={0: recent_state(wl, 0, 14)}, independent=False)
    say(f"stress: {s}")


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
