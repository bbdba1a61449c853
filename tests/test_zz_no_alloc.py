"""skv_frame_step_noalloc (per-call scratch in the library's static device array)
against skv_frame_step on the same inputs, through the C ABI.

Two workloads in a row, the second smaller: the 7B-shaped single layer (one call
per frame; a key-split plan, so the scratch holds row statistics and output shares
besides the column-sum partials) and then a two-layer stack of small heads stepped
one layer per call.  Every call's output, state (slots, positions, scores), pool
scores and decode-cache rows must equal the allocating entry point's bit for bit.
A call whose scratch exceeds the static array is refused before anything is
enqueued.
"""
from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2605_31598_amd import FrameStepper, StateKVError  # noqa: E402
from paper_2605_31598_amd import binding as B  # noqa: E402
from workloads import WorkloadConfig  # noqa: E402

from .gpu_harness import frame_tensors, say  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


def _compare(ref, got, wl, where):
    for l in range(wl.n_layers):
        a, b = ref.read_state(l), got.read_state(l)
        for key in ("pos", "score", "k", "v", "pool_score", "pool_pos"):
            assert np.array_equal(a[key], b[key]), f"{where}: {key} of layer {l}"
        ca, cb = ref.read_cache(l), got.read_cache(l)
        assert ca[2] == cb[2] and np.array_equal(ca[0], cb[0]) and np.array_equal(ca[1], cb[1]), \
            f"{where}: decode cache of layer {l}"


def _run(wl, per_layer):
    ref = FrameStepper.from_workload(wl)
    got = FrameStepper.from_workload(wl)
    L, Hq, T, d = wl.n_layers, wl.n_q_heads, wl.tokens_per_frame, wl.head_dim
    try:
        o_ref = torch.empty((L, Hq, T, d), dtype=torch.bfloat16, device="cuda")
        o_got = torch.full_like(o_ref, 7.0)
        for n in range(wl.n_frames):
            q, k, v, _ = frame_tensors(wl, n, list(range(L)))
            spans = [(l, 1) for l in range(L)] if per_layer else [(0, L)]
            for l0, lc in spans:
                sl = slice(l0, l0 + lc)
                ref.step(q[sl], k[sl], v[sl], o_ref[sl], layer_begin=l0, layer_count=lc)
                B.skv_frame_step_noalloc(got.ctx, l0, lc, q[sl].data_ptr(), k[sl].data_ptr(), v[sl].data_ptr(),
                                         o_got[sl].data_ptr())
            torch.cuda.synchronize()
            assert torch.equal(o_ref.view(torch.int16), o_got.view(torch.int16)), f"{wl.name} frame {n}: output"
            _compare(ref, got, wl, f"{wl.name} frame {n}")
        say(f"{wl.name}: {wl.n_frames} frames equal, {'one layer' if per_layer else 'all layers'} per call")
    finally:
        ref.close()
        got.close()


def test_noalloc_matches_frame_step_two_calls_second_smaller():
    _run(WorkloadConfig("noalloc_7b_layer", 1, 28, 4, 128, 196, 8, 1024, "bf16", "iid", 8080, pos_offset=3), False)
    _run(WorkloadConfig("noalloc_small", 2, 8, 2, 64, 40, 5, 64, "bf16", "iid", 8081), True)


def test_noalloc_refuses_calls_beyond_its_scratch():
    # 40 layers x 8 KV heads of 2048 query rows over pools of 4352 candidates: the
    # column-sum partials alone exceed 64 MiB
    wl = WorkloadConfig("noalloc_big", 40, 64, 8, 128, 256, 1, 4096, "bf16", "iid", 8082)
    st = FrameStepper.from_workload(wl)
    try:
        q, k, v, _ = frame_tensors(wl, 0, [])
        out = torch.empty_like(q)
        with pytest.raises(StateKVError, match="SKV_ERR_UNSUPPORTED.*scratch"):
            B.skv_frame_step_noalloc(st.ctx, 0, wl.n_layers, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                     out.data_ptr())
        assert st.read_state(0)["frame"] == 0  # nothing happened
        B.skv_frame_step_noalloc(st.ctx, 0, 1, q[:1].data_ptr(), k[:1].data_ptr(), v[:1].data_ptr(),
                                 out[:1].data_ptr())  # one layer fits
        torch.cuda.synchronize()
        assert st.read_state(0)["frame"] == 1
    finally:
        st.close()
