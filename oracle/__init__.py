"""CPU oracle for the StateKV per-frame video-prefill step.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg; never by the GPU library.  Every function is
pinned by the ``-m "not gpu"`` tests (brute force, closed forms, library
routines, invariants, a hand-derived worked example).
"""
from .statekv_oracle import (  # noqa: F401
    DecodeCache,
    LayerState,
    StepResult,
    attention_flops,
    frame_attention,
    frame_positions,
    frame_step,
    importance_scores,
    kv_head_of,
    run_layer,
    select_top,
    visibility,
)
