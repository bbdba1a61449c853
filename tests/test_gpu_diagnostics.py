"""GPU run of the assumption diagnostics against the fp64 oracle.

A 16-frame stream at the 7B one-layer shape with a capacity that keeps every
token, so each frame's importance scores cover its whole history.  The layer
scores from the library (summed over KV heads) must match the oracle's within
1e-3 relative, and the diagnostics computed from both within 2e-3
(concentration) and 0.05 (set-based recall / retention / churn, which a
near-tie between the B-th and (B+1)-th key can move by 1/B).
"""
import numpy as np
import pytest
import torch

from oracle import statekv_oracle as orc
from paper_2605_31598_amd import FrameStepper
from paper_2605_31598_amd import diagnostics as dg
from workloads import CONFIGS

from .gpu_harness import frame_tensors, say, widen

pytestmark = pytest.mark.gpu


def test_diagnostics_match_the_oracle():
    n_frames = 16
    wl = CONFIGS["vlm7b_1layer"]
    wl = wl.with_(capacity=n_frames * wl.tokens_per_frame)
    T = wl.tokens_per_frame
    st = FrameStepper.from_workload(wl, max_frames=n_frames)
    state = orc.LayerState.empty(wl.n_kv_heads, wl.head_dim)
    out = torch.empty((1, wl.n_q_heads, T, wl.head_dim), dtype=torch.bfloat16, device="cuda")
    gpu_frames, orc_frames = [], []
    try:
        for n in range(n_frames):
            q, k, v, host = frame_tensors(wl, n, [0])
            st.step(q, k, v, out)
            s_gpu, p_gpu = dg.layer_frames_from_stepper(st, 0, T)
            x = host[0]
            r = orc.frame_step(state, widen(x["q"], "bf16"), widen(x["k"], "bf16"), widen(x["v"], "bf16"), n,
                               wl.capacity, wl.scale, wl.pos_offset)
            state = r.state
            s_orc = r.pool_score.sum(axis=0) * T
            p_orc = r.pool_pos[0]
            o = np.argsort(p_gpu)
            assert np.array_equal(p_gpu[o], p_orc)
            rel = np.abs(s_gpu[o] - s_orc) / s_orc
            assert rel.max() <= 1e-3, f"frame {n}: layer score rel {rel.max():.3e}"
            f0 = wl.pos_offset + n * T
            gpu_frames.append((s_gpu, p_gpu, f0))
            orc_frames.append((s_orc, p_orc, f0))
    finally:
        st.close()
    budgets = [16, 256, 1024]
    g = dg.summarise(gpu_frames, budgets)
    o = dg.summarise(orc_frames, budgets)
    for b in budgets:
        say(f"B={b}: gpu {g[b]}")
        assert abs(g[b]["concentration"] - o[b]["concentration"]) <= 2e-3
        for key in ("recall", "weighted_recall", "retention", "churn"):
            assert abs(g[b][key] - o[b][key]) <= 0.05, f"B={b} {key}: {g[b][key]} vs {o[b][key]}"
