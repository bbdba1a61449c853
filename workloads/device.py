"""Device-side filling of generator streams (benchmark inputs in HBM).

Same definition as ``workloads.generate`` (SplitMix64 counter hash + uploaded
quantile table), implemented in workloads/csrc/skv_gen.hip: the i.i.d. streams,
and the low-rank and stress key recipes built from those streams.
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


def fill_lowrank_keys(out, cfg, layer: int, frames, stream=None):
    """Low-rank keys of one layer for ``frames``: ``out`` is a bf16 CUDA tensor
    [len(frames), H_kv, T, d].  Bit-identical to ``generate.frame_inputs(...)["k"]``:
    the same fp32 streams, the rank-one terms multiplied and added one at a time
    (no fused multiply-add), then scaled and rounded to bf16 the same way."""
    import torch

    H, T, d, R = cfg.n_kv_heads, cfg.tokens_per_frame, cfg.head_dim, gen.LOWRANK_RANK
    F = len(frames)
    dev = out.device
    W = torch.empty((1, H * R * d), dtype=torch.float32, device=dev)
    fill_iid(W, [gen.stream_key(cfg.seed, layer, 0, gen.TENSOR_LOWRANK_W)], "f32", stream)
    c = torch.empty((F, H * T * R), dtype=torch.float32, device=dev)
    fill_iid(c, [gen.stream_key(cfg.seed, layer, f, gen.TENSOR_LOWRANK_C) for f in frames], "f32", stream)
    eps = torch.empty((F, H * T * d), dtype=torch.float32, device=dev)
    fill_iid(eps, [gen.stream_key(cfg.seed, layer, f, gen.TENSOR_K) for f in frames], "f32", stream)
    W = W.view(H, R, d)
    c = c.view(F, H, T, R)
    acc = torch.zeros((F, H, T, d), dtype=torch.float32, device=dev)
    for r in range(R):
        prod = c[:, :, :, r:r + 1] * W[None, :, r, None, :]
        acc = acc + prod
    val = acc * 0.25 + eps.view(F, H, T, d) * 0.5
    out.copy_(val.to(torch.bfloat16))


def fill_stress_keys(out, cfg, layer: int, frames, stream=None):
    """Stress keys of one layer for ``frames``: ``out`` is a bf16 CUDA tensor
    [len(frames), H_kv, T, d].  Bit-identical to ``generate.frame_inputs(...)["k"]``
    for the stress recipe: the i.i.d. key stream, then per (frame, KV head) the tokens
    ranked n_heavy..n_heavy+n_dup-1 by the rank stream copy a template row (picked by
    the pick stream) and the first n_heavy are multiplied by 4 (exact in bf16).  The
    ranking is done on the host from the same counter streams."""
    import torch

    H, T, d = cfg.n_kv_heads, cfg.tokens_per_frame, cfg.head_dim
    frames = list(frames)
    F = len(frames)
    dev = out.device
    fill_iid(out.view(F, H * T * d), [gen.stream_key(cfg.seed, layer, f, gen.TENSOR_K) for f in frames], "bf16",
             stream)
    tmpl = torch.empty((1, H * gen.STRESS_TEMPLATES * d), dtype=torch.bfloat16, device=dev)
    fill_iid(tmpl, [gen.stream_key(cfg.seed, layer, 0, gen.TENSOR_STRESS_TMPL)], "bf16", stream)
    tmpl = tmpl.view(H, gen.STRESS_TEMPLATES, d)
    n_heavy = int(round(gen.STRESS_HEAVY_FRACTION * T))
    n_dup = int(round(gen.STRESS_DUP_FRACTION * T))
    dup_idx, heavy_idx = [], []
    heads = np.arange(H)[:, None]
    for i, f in enumerate(frames):
        rank = gen.raw_bits(gen.stream_key(cfg.seed, layer, f, gen.TENSOR_STRESS_RANK), H * T).reshape(H, T)
        pick = gen.raw_bits(gen.stream_key(cfg.seed, layer, f, gen.TENSOR_STRESS_PICK), H * T).reshape(H, T)
        order = np.argsort(rank, axis=1, kind="stable")
        dup = order[:, n_heavy:n_heavy + n_dup]
        src = (pick[heads, dup] % np.uint64(gen.STRESS_TEMPLATES)).astype(np.int64)
        g = np.broadcast_to(heads, dup.shape)
        dup_idx.append(np.stack([np.full(dup.size, i), g.ravel(), dup.ravel(), src.ravel()]))
        hv = order[:, :n_heavy]
        heavy_idx.append(np.stack([np.full(hv.size, i), np.broadcast_to(heads, hv.shape).ravel(), hv.ravel()]))
    k = out.view(F, H, T, d)
    di = torch.from_numpy(np.concatenate(dup_idx, axis=1)).to(dev)
    k[di[0], di[1], di[2]] = tmpl[di[1], di[3]]
    hi = torch.from_numpy(np.concatenate(heavy_idx, axis=1)).to(dev)
    k[hi[0], hi[1], hi[2]] = k[hi[0], hi[1], hi[2]] * 4.0
