"""ctypes binding of libstatekv.so (C ABI in include/statekv.h).

Argument marshalling only: every step of the frame step runs in the library's
HIP kernels.  Importing this module does not need a GPU; loading the library
fails loudly if it has not been built.  PyTorch is used by callers for device
memory and streams; here only raw device pointers and HIP copies are handled.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libstatekv.so")

SKV_OK = 0
SKV_ERR_INVALID_ARG = -1
SKV_ERR_OUT_OF_MEMORY = -2
SKV_ERR_CAPACITY = -3
SKV_ERR_ORDER = -4
SKV_ERR_DEVICE = -5
SKV_ERR_UNSUPPORTED = -6

SKV_BF16 = 0
SKV_F32 = 1

SKV_POLICY_STATEKV = 0
SKV_POLICY_RECENT = 1
SKV_POLICY_FULL = 2
POLICIES = {"statekv": SKV_POLICY_STATEKV, "recent": SKV_POLICY_RECENT, "full": SKV_POLICY_FULL}

SKV_ROPE_NONE = 0
SKV_ROPE_PLAIN = 1
SKV_ROPE_YARN = 2
N_STAGES = 4
STAGES = ("attention", "refresh", "state_update", "append")

# Every symbol declared in include/statekv.h.
EXPORTS = (
    "skv_init", "skv_frame_step", "skv_frame_step_noalloc", "skv_decode_step", "skv_state_view",
    "skv_decode_cache_view", "skv_reset", "skv_seek",
    "skv_timing_start", "skv_timing_stride", "skv_timing_stop", "skv_destroy", "skv_status_string", "skv_last_error",
)


class skv_config(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("tokens_per_frame", ctypes.c_int32), ("capacity", ctypes.c_int32),
        ("max_frames", ctypes.c_int32), ("dtype", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
        ("pos_offset", ctypes.c_int64), ("policy", ctypes.c_int32), ("max_decode_tokens", ctypes.c_int32),
        ("rope", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("rope_factor", ctypes.c_float),
        ("rope_orig_max", ctypes.c_int32), ("split_refresh", ctypes.c_int32),
        ("key_split_mode", ctypes.c_int32),
    ]


class skv_state_view_t(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("pos", ctypes.c_void_p), ("score", ctypes.c_void_p),
        ("size", ctypes.c_int32), ("capacity", ctypes.c_int32), ("frame", ctypes.c_int64),
        ("pool_score", ctypes.c_void_p), ("pool_pos", ctypes.c_void_p), ("pool_size", ctypes.c_int32),
        ("pool_stride", ctypes.c_int32),
    ]


class skv_cache_view_t(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("n_tokens", ctypes.c_int64), ("max_tokens", ctypes.c_int64),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("decode_row0", ctypes.c_int64),
        ("decode_tokens", ctypes.c_int64),
    ]


class StateKVError(RuntimeError):
    def __init__(self, status, where, detail):
        self.status = status
        super().__init__(f"{where}: {detail}")


_lib = None
_hip = None


def load_library(path: str = LIB_PATH):
    """Load libstatekv.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(python paper_2605_31598_amd/build.py)")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.skv_init.argtypes = [P(skv_config), ctypes.c_void_p, P(ctypes.c_void_p)]
    lib.skv_frame_step.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.skv_frame_step_noalloc.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.skv_decode_step.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.skv_state_view.argtypes = [ctypes.c_void_p, ctypes.c_int32, P(skv_state_view_t)]
    lib.skv_decode_cache_view.argtypes = [ctypes.c_void_p, ctypes.c_int32, P(skv_cache_view_t)]
    lib.skv_reset.argtypes = [ctypes.c_void_p]
    lib.skv_seek.argtypes = [ctypes.c_void_p, ctypes.c_int64]
    lib.skv_timing_start.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    lib.skv_timing_stride.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    lib.skv_timing_stop.argtypes = [ctypes.c_void_p, P(ctypes.c_int32), P(ctypes.c_float), ctypes.c_int32]
    lib.skv_destroy.argtypes = [ctypes.c_void_p]
    lib.skv_destroy.restype = None
    lib.skv_status_string.argtypes = [ctypes.c_int]
    lib.skv_status_string.restype = ctypes.c_char_p
    lib.skv_last_error.argtypes = []
    lib.skv_last_error.restype = ctypes.c_char_p
    for name in ("skv_init", "skv_frame_step", "skv_frame_step_noalloc", "skv_decode_step", "skv_state_view",
                 "skv_decode_cache_view", "skv_reset",
                 "skv_seek", "skv_timing_start", "skv_timing_stride", "skv_timing_stop"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _hip_runtime():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
        _hip.hipDeviceSynchronize.restype = ctypes.c_int
    return _hip


def _check(status, where):
    if status != SKV_OK:
        lib = load_library()
        name = lib.skv_status_string(status).decode()
        detail = lib.skv_last_error().decode()
        raise StateKVError(status, where, f"{name}: {detail}")


def status_string(status: int) -> str:
    return load_library().skv_status_string(status).decode()


def skv_init(cfg: skv_config, stream: int = 0) -> int:
    lib = load_library()
    h = ctypes.c_void_p()
    _check(lib.skv_init(ctypes.byref(cfg), ctypes.c_void_p(stream), ctypes.byref(h)), "skv_init")
    return h.value


def skv_frame_step(ctx: int, layer_begin: int, layer_count: int, q: int, k: int, v: int, out: int) -> None:
    _check(load_library().skv_frame_step(ctypes.c_void_p(ctx), layer_begin, layer_count, ctypes.c_void_p(q),
                                         ctypes.c_void_p(k), ctypes.c_void_p(v), ctypes.c_void_p(out)),
           "skv_frame_step")


def skv_frame_step_noalloc(ctx: int, layer_begin: int, layer_count: int, q: int, k: int, v: int, out: int) -> None:
    _check(load_library().skv_frame_step_noalloc(ctypes.c_void_p(ctx), layer_begin, layer_count, ctypes.c_void_p(q),
                                                 ctypes.c_void_p(k), ctypes.c_void_p(v), ctypes.c_void_p(out)),
           "skv_frame_step_noalloc")


def skv_decode_step(ctx: int, layer_begin: int, layer_count: int, n_tokens: int, q: int, k: int, v: int,
                    out: int) -> None:
    _check(load_library().skv_decode_step(ctypes.c_void_p(ctx), layer_begin, layer_count, n_tokens,
                                          ctypes.c_void_p(q), ctypes.c_void_p(k), ctypes.c_void_p(v),
                                          ctypes.c_void_p(out)),
           "skv_decode_step")


def skv_state_view(ctx: int, layer: int) -> skv_state_view_t:
    out = skv_state_view_t()
    _check(load_library().skv_state_view(ctypes.c_void_p(ctx), layer, ctypes.byref(out)), "skv_state_view")
    return out


def skv_decode_cache_view(ctx: int, layer: int) -> skv_cache_view_t:
    out = skv_cache_view_t()
    _check(load_library().skv_decode_cache_view(ctypes.c_void_p(ctx), layer, ctypes.byref(out)),
           "skv_decode_cache_view")
    return out


def skv_reset(ctx: int) -> None:
    _check(load_library().skv_reset(ctypes.c_void_p(ctx)), "skv_reset")


def skv_seek(ctx: int, frame: int) -> None:
    _check(load_library().skv_seek(ctypes.c_void_p(ctx), frame), "skv_seek")


def skv_timing_start(ctx: int, max_steps: int) -> None:
    _check(load_library().skv_timing_start(ctypes.c_void_p(ctx), max_steps), "skv_timing_start")


def skv_timing_stride(ctx: int, stride: int) -> None:
    _check(load_library().skv_timing_stride(ctypes.c_void_p(ctx), stride), "skv_timing_stride")


def skv_timing_stop(ctx: int, max_steps: int) -> np.ndarray:
    """Per-step stage times in ms, shape [n_steps, N_STAGES]: attention, refresh (with
    split_refresh: the selection launch), state update and append (split_refresh only;
    a decode step fills attention and append)."""
    buf = (ctypes.c_float * (max_steps * N_STAGES))()
    n = ctypes.c_int32(0)
    _check(load_library().skv_timing_stop(ctypes.c_void_p(ctx), ctypes.byref(n), buf, max_steps * N_STAGES),
           "skv_timing_stop")
    return np.frombuffer(buf, dtype=np.float32, count=n.value * N_STAGES).reshape(n.value, N_STAGES).copy()


def skv_destroy(ctx: int) -> None:
    if ctx:
        load_library().skv_destroy(ctypes.c_void_p(ctx))


# ---------------------------------------------------------------------------
# Device <-> host copies of the borrowed views (test and benchmark plumbing).
# The caller synchronises the library's stream first; hipMemcpy is blocking.
# ---------------------------------------------------------------------------
def copy_to_host(ptr: int, nbytes: int) -> np.ndarray:
    out = np.empty(nbytes, dtype=np.uint8)
    if nbytes:
        err = _hip_runtime().hipMemcpy(out.ctypes.data, ctypes.c_void_p(ptr), nbytes, 2)
        if err != 0:
            raise RuntimeError(f"hipMemcpy device->host failed: {err}")
    return out


def copy_to_device(ptr: int, data: np.ndarray) -> None:
    data = np.ascontiguousarray(data)
    if data.nbytes:
        err = _hip_runtime().hipMemcpy(ctypes.c_void_p(ptr), data.ctypes.data, data.nbytes, 1)
        if err != 0:
            raise RuntimeError(f"hipMemcpy host->device failed: {err}")
