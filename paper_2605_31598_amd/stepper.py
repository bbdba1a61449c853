"""Python front end of one StateKV video stream on the GPU.

Thin layer over the C ABI: checks tensor shapes/dtypes/devices, passes raw
pointers and the torch stream to the library, and copies the borrowed state
and decode-cache views to or from the host.  All arithmetic of the step runs
in the library's HIP kernels.
"""
from __future__ import annotations

import numpy as np

from . import binding as B

_DTYPES = {"bf16": B.SKV_BF16, "f32": B.SKV_F32}


class FrameStepper:
    """One video stream: compressed state and decode cache of every layer."""

    def __init__(self, n_layers, n_q_heads, n_kv_heads, head_dim, tokens_per_frame, capacity, max_frames,
                 dtype="bf16", softmax_scale=0.0, pos_offset=0, stream=None, policy="statekv",
                 max_decode_tokens=0, rope=None, rope_theta=0.0, rope_factor=1.0, rope_orig_max=0,
                 split_refresh=False, key_split_mode=0):
        import torch

        if not torch.cuda.is_available():
            raise RuntimeError("FrameStepper needs a ROCm GPU (torch.cuda.is_available() is False)")
        self.torch = torch
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self.dtype = dtype
        self.torch_dtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.np_dtype = np.uint16 if dtype == "bf16" else np.float32
        self.elem = 2 if dtype == "bf16" else 4
        self.policy = policy
        self.cfg = B.skv_config(n_layers, n_q_heads, n_kv_heads, head_dim, tokens_per_frame, capacity, max_frames,
                                _DTYPES[dtype], softmax_scale, pos_offset, B.POLICIES[policy], max_decode_tokens,
                                {None: B.SKV_ROPE_NONE, "plain": B.SKV_ROPE_PLAIN, "yarn": B.SKV_ROPE_YARN}[rope],
                                rope_theta, rope_factor, rope_orig_max, int(bool(split_refresh)), int(key_split_mode))
        self.n_layers, self.H_q, self.H_kv, self.d = n_layers, n_q_heads, n_kv_heads, head_dim
        # streaming full attention keeps no compressed state
        self.T, self.B, self.max_frames = tokens_per_frame, (0 if policy == "full" else capacity), max_frames
        self.ctx = B.skv_init(self.cfg, self.stream.cuda_stream)

    @classmethod
    def from_workload(cls, wl, max_frames=None, stream=None, policy="statekv", max_decode_tokens=0, **kw):
        return cls(wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.tokens_per_frame, wl.capacity,
                   max_frames or wl.n_frames, wl.dtype, 0.0, wl.pos_offset, stream, policy, max_decode_tokens, **kw)

    # ------------------------------------------------------------------ step
    def _check(self, name, t, heads, n_layers):
        if t.device.type != "cuda" or t.dtype != self.torch_dtype or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {self.torch_dtype} CUDA tensor")
        if t.numel() != n_layers * heads * self.T * self.d:
            raise ValueError(f"{name} has {t.numel()} elements, expected [{n_layers}][{heads}][{self.T}][{self.d}]")

    def step(self, q, k, v, out, layer_begin=0, layer_count=None):
        lc = self.n_layers - layer_begin if layer_count is None else layer_count
        self._check("q", q, self.H_q, lc)
        self._check("k", k, self.H_kv, lc)
        self._check("v", v, self.H_kv, lc)
        self._check("out", out, self.H_q, lc)
        B.skv_frame_step(self.ctx, layer_begin, lc, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr())

    def decode(self, q, k, v, out, layer_begin=0, layer_count=None):
        """Decode step over the detailed cache: q/out [layers][H_q][t][d], k/v [layers][H_kv][t][d]."""
        lc = self.n_layers - layer_begin if layer_count is None else layer_count
        t = q.shape[-2]
        for name, x, heads in (("q", q, self.H_q), ("k", k, self.H_kv), ("v", v, self.H_kv), ("out", out, self.H_q)):
            if x.device.type != "cuda" or x.dtype != self.torch_dtype or not x.is_contiguous():
                raise ValueError(f"{name} must be a contiguous {self.torch_dtype} CUDA tensor")
            if x.numel() != lc * heads * t * self.d:
                raise ValueError(f"{name} has {x.numel()} elements, expected [{lc}][{heads}][{t}][{self.d}]")
        B.skv_decode_step(self.ctx, layer_begin, lc, t, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr())

    def read_decode_rows(self, layer):
        """Host copy of the decode rows of one layer's cache: (k, v) [H_kv, n, d]."""
        self._sync()
        cv = B.skv_decode_cache_view(self.ctx, layer)
        H, d, M, n, r0 = self.H_kv, self.d, cv.max_tokens, cv.decode_tokens, cv.decode_row0
        out = []
        for base in (cv.k, cv.v):
            arr = np.empty((H, n, d), dtype=self.np_dtype)
            for g in range(H):
                arr[g] = B.copy_to_host(base + (g * M + r0) * d * self.elem, n * d * self.elem).view(
                    self.np_dtype).reshape(n, d)
            out.append(arr)
        return out[0], out[1]

    def reset(self):
        B.skv_reset(self.ctx)

    def seek(self, frame):
        B.skv_seek(self.ctx, frame)

    # ------------------------------------------------------------- views
    def _sync(self):
        self.stream.synchronize()

    def read_state(self, layer):
        """Host copy of one layer's compressed state and last candidate pool."""
        sv = B.skv_state_view(self.ctx, layer)  # enqueues a deferred selection, if any
        self._sync()
        H, cap, d, n = self.H_kv, self.B, self.d, sv.size
        kb = B.copy_to_host(sv.k, H * cap * d * self.elem).view(self.np_dtype).reshape(H, cap, d)
        vb = B.copy_to_host(sv.v, H * cap * d * self.elem).view(self.np_dtype).reshape(H, cap, d)
        pos = B.copy_to_host(sv.pos, H * cap * 4).view(np.int32).reshape(H, cap)
        score = B.copy_to_host(sv.score, H * cap * 4).view(np.float32).reshape(H, cap)
        ps = B.copy_to_host(sv.pool_score, H * sv.pool_stride * 4).view(np.float32).reshape(H, sv.pool_stride)
        pp = B.copy_to_host(sv.pool_pos, H * sv.pool_stride * 4).view(np.int32).reshape(H, sv.pool_stride)
        return {
            "k": kb[:, :n], "v": vb[:, :n], "pos": pos[:, :n], "score": score[:, :n], "size": n,
            "frame": sv.frame, "pool_score": ps[:, :sv.pool_size], "pool_pos": pp[:, :sv.pool_size],
        }

    def write_state(self, layer, pos, k, v, score=None):
        """Overwrite slots 0..n-1 of every KV head (n = pos.shape[1]) to force a state."""
        sv = B.skv_state_view(self.ctx, layer)  # enqueues a deferred selection, if any
        self._sync()
        H, cap, d = self.H_kv, self.B, self.d
        n = pos.shape[1]
        if n != sv.size:
            raise ValueError(f"state of layer {layer} holds {sv.size} entries at this frame, got {n}")
        kb = np.zeros((H, cap, d), dtype=self.np_dtype)
        vb = np.zeros((H, cap, d), dtype=self.np_dtype)
        pb = np.zeros((H, cap), dtype=np.int32)
        sb = np.zeros((H, cap), dtype=np.float32)
        kb[:, :n] = k
        vb[:, :n] = v
        pb[:, :n] = pos
        if score is not None:
            sb[:, :n] = score
        B.copy_to_device(sv.k, kb)
        B.copy_to_device(sv.v, vb)
        B.copy_to_device(sv.pos, pb)
        B.copy_to_device(sv.score, sb)

    def read_cache(self, layer, rows=None):
        self._sync()
        cv = B.skv_decode_cache_view(self.ctx, layer)
        n = cv.n_tokens if rows is None else rows
        H, d, M = self.H_kv, self.d, cv.max_tokens
        out = []
        for base in (cv.k, cv.v):
            arr = np.empty((H, n, d), dtype=self.np_dtype)
            for g in range(H):
                arr[g] = B.copy_to_host(base + g * M * d * self.elem, n * d * self.elem).view(self.np_dtype).reshape(n, d)
            out.append(arr)
        return out[0], out[1], cv.n_tokens

    def read_cache_rows(self, layer, r0, r1):
        """Host copy of decode-cache rows [r0, r1) of every KV head: (k, v) [H_kv, r1 - r0, d]
        and the number of video rows the layer has written."""
        self._sync()
        cv = B.skv_decode_cache_view(self.ctx, layer)
        H, d, M, n = self.H_kv, self.d, cv.max_tokens, r1 - r0
        if not 0 <= r0 <= r1 <= M:
            raise ValueError(f"rows [{r0}, {r1}) outside the cache's {M} rows")
        out = []
        for base in (cv.k, cv.v):
            arr = np.empty((H, n, d), dtype=self.np_dtype)
            for g in range(H):
                arr[g] = B.copy_to_host(base + (g * M + r0) * d * self.elem, n * d * self.elem).view(
                    self.np_dtype).reshape(n, d)
            out.append(arr)
        return out[0], out[1], cv.n_tokens

    def write_cache(self, layer, k, v):
        """Overwrite decode-cache rows 0..n-1 of every KV head (k, v [H_kv, n, d] in storage
        form), e.g. to give a streaming-full-attention step a history without running it."""
        self._sync()
        cv = B.skv_decode_cache_view(self.ctx, layer)
        H, d, M = self.H_kv, self.d, cv.max_tokens
        n = k.shape[1]
        if k.shape != (H, n, d) or v.shape != (H, n, d) or n > M:
            raise ValueError(f"cache rows must be [{H}][n <= {M}][{d}]")
        for base, arr in ((cv.k, k), (cv.v, v)):
            for g in range(H):
                B.copy_to_device(base + g * M * d * self.elem, np.ascontiguousarray(arr[g], dtype=self.np_dtype))

    # ------------------------------------------------------------ timing
    def timing_start(self, max_steps, stride=1):
        """Record stage events on the next max_steps steps, or with stride > 1 on every
        stride-th step (the first, stride + 1-th, ...) until max_steps are recorded."""
        B.skv_timing_start(self.ctx, max_steps)
        if stride != 1:
            B.skv_timing_stride(self.ctx, stride)

    def timing_stop(self, max_steps):
        return B.skv_timing_stop(self.ctx, max_steps)

    def close(self):
        if getattr(self, "ctx", None):
            self._sync()
            B.skv_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
