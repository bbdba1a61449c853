"""Device-side filling of generator streams (benchmark inputs in HBM).

Same definition as ``workloads.generate`` (SplitMix64 counter hash + uploaded
quantile table), implemented in workloads/csrc/skv_gen.hip.  Only the i.i.d.
recipe is provided on the device.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import generate as gen

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libskvgen.so")
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} missing: build with __graft_entry__.build()")
        _lib = ctypes.CDLL(LIB_PATH)
        _lib.skvgen_fill.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
        _lib.skvgen_fill.restype = ctypes.c_int
    return _lib


def fill_iid(out, keys, dtype: str, stream=None):
    """Fill torch CUDA tensor ``out`` (len(keys) equal chunks) with the i.i.d. streams of ``keys``."""
    import torch

    n_chunks = len(keys)
    if out.numel() % n_chunks:
        raise ValueError("output does not split into equal chunks")
    stream = stream or torch.cuda.current_stream()
    table = gen.normal_table(dtype)
    tbl = torch.from_numpy(table.view(np.int16) if dtype == "bf16" else table.copy()).to(out.device)
    kd = torch.from_numpy(np.array(keys, dtype=np.uint64).view(np.int64)).to(out.device)
    err = _load().skvgen_fill(out.data_ptr(), out.numel() // n_chunks, n_chunks, kd.data_ptr(), tbl.data_ptr(),
                              2 if dtype == "bf16" else 4, ctypes.c_void_p(stream.cuda_stream))
    if err != 0:
        raise RuntimeError(f"skvgen_fill failed: {err}")
    stream.synchronize()  # keeps the uploaded keys/table alive until the kernel has read them
