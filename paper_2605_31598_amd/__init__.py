"""StateKV per-frame streaming video-prefill step on AMD Instinct MI355X (gfx950).

The step runs in libstatekv.so (hand-written HIP kernels, C ABI in
include/statekv.h).  ``binding`` mirrors the C entry points one to one;
``FrameStepper`` is a thin front end that takes torch device tensors.
"""
from .binding import (  # noqa: F401
    EXPORTS,
    LIB_PATH,
    StateKVError,
    load_library,
    skv_config,
    skv_decode_cache_view,
    skv_destroy,
    skv_frame_step,
    skv_init,
    skv_reset,
    skv_seek,
    skv_state_view,
    skv_timing_start,
    skv_timing_stop,
)
from .stepper import FrameStepper  # noqa: F401
