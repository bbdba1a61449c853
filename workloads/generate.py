"""Deterministic, counter-based input generator (host side).

Every value is a pure function of (seed, layer, frame, tensor id, flat index),
so any slice of a video can be produced independently and a device
implementation of the same definition produces the same bytes.

Definition
----------
* ``mix64`` is the SplitMix64 output function (Steele, Lea & Flood,
  "Fast splittable pseudorandom number generators", OOPSLA 2014):
  ``z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27; z *= 0x94D049BB133111EB;
  z ^= z >> 31`` on 64-bit unsigned integers.
* A stream key is ``mix64(mix64(mix64(seed) ^ (layer << 32 | frame)) ^ tensor)``.
* Element ``i`` of a stream draws ``bits = mix64(key + (i + 1) * 0x9E3779B97F4A7C15)``
  and takes the top 16 bits as an index into a 65,536-entry table of standard
  normal quantiles ``Phi^-1((i + 1/2) / 65536)``, rounded once to the storage
  type (fp32, or bf16 with round-to-nearest-even).  No floating-point arithmetic
  happens per element, so host and device agree bit for bit.

bf16 tensors are carried as ``uint16`` bit patterns; ``bf16_to_f64`` widens them
exactly.  This module holds no part of the attention/scoring/selection method.
"""
from __future__ import annotations

import functools

import numpy as np

from .configs import WorkloadConfig

GOLDEN = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB
_MASK = (1 << 64) - 1

# Tensor ids of the per-(layer, frame) streams.
TENSOR_Q = 1
TENSOR_K = 2
TENSOR_V = 3
TENSOR_LOWRANK_W = 4  # per-(layer) rank-16 basis, frame field fixed at 0
TENSOR_LOWRANK_C = 5  # per-token rank-16 coefficients
TENSOR_STRESS_RANK = 6  # per-(frame, kv head) ordering of tokens
TENSOR_STRESS_TMPL = 7  # per-(layer) template key rows, frame field fixed at 0
TENSOR_STRESS_PICK = 8  # which template a duplicated token copies

LOWRANK_RANK = 16
STRESS_TEMPLATES = 32
STRESS_HEAVY_FRACTION = 0.02
STRESS_DUP_FRACTION = 0.10
STRESS_HEAVY_MULT = 4.0


def mix64_int(z: int) -> int:
    z &= _MASK
    z = ((z ^ (z >> 30)) * _M1) & _MASK
    z = ((z ^ (z >> 27)) * _M2) & _MASK
    return z ^ (z >> 31)


def mix64(z: np.ndarray) -> np.ndarray:
    z = z.astype(np.uint64, copy=True)
    with np.errstate(over="ignore"):
        z ^= z >> np.uint64(30)
        z *= np.uint64(_M1)
        z ^= z >> np.uint64(27)
        z *= np.uint64(_M2)
        z ^= z >> np.uint64(31)
    return z


def stream_key(seed: int, layer: int, frame: int, tensor: int) -> int:
    k = mix64_int(seed)
    k = mix64_int(k ^ (((layer & 0xFFFFFFFF) << 32) | (frame & 0xFFFFFFFF)))
    return mix64_int(k ^ tensor)


def raw_bits(key: int, n: int, start: int = 0) -> np.ndarray:
    idx = np.arange(start + 1, start + n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(key) + idx * np.uint64(GOLDEN)
    return mix64(z)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))
    return (b >> np.uint64(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return bf16_to_f32(bits).astype(np.float64)


@functools.lru_cache(maxsize=None)
def normal_table(dtype: str) -> np.ndarray:
    """65,536 standard-normal quantiles at cell midpoints, rounded to ``dtype``."""
    from scipy.special import ndtri

    p = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
    x = ndtri(p).astype(np.float32)
    if dtype == "f32":
        out = x
    elif dtype == "bf16":
        out = f32_to_bf16_bits(x)
    else:
        raise ValueError(dtype)
    out.setflags(write=False)
    return out


def iid(key: int, shape, dtype: str) -> np.ndarray:
    n = int(np.prod(shape))
    table = normal_table(dtype)
    return table[(raw_bits(key, n) >> np.uint64(48)).astype(np.int64)].reshape(shape)


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_to_f64(x) if dtype == "bf16" else np.asarray(x, dtype=np.float64)


def _lowrank_keys(cfg: WorkloadConfig, layer: int, frame: int) -> np.ndarray:
    """K = bf16(fl32(c.W) / 4 + 0.5 * eps) with c, W, eps standard normal (fp32 table)."""
    H, T, d, R = cfg.n_kv_heads, cfg.tokens_per_frame, cfg.head_dim, LOWRANK_RANK
    W = iid(stream_key(cfg.seed, layer, 0, TENSOR_LOWRANK_W), (H, R, d), "f32")
    c = iid(stream_key(cfg.seed, layer, frame, TENSOR_LOWRANK_C), (H, T, R), "f32")
    eps = iid(stream_key(cfg.seed, layer, frame, TENSOR_K), (H, T, d), "f32")
    acc = np.zeros((H, T, d), dtype=np.float32)
    for r in range(R):  # fixed order, separate fp32 multiply and add (no fused multiply-add)
        prod = (c[:, :, r:r + 1] * W[:, None, r, :]).astype(np.float32)
        acc = (acc + prod).astype(np.float32)
    val = (acc * np.float32(0.25)).astype(np.float32) + (eps * np.float32(0.5)).astype(np.float32)
    return f32_to_bf16_bits(val.astype(np.float32))


def _stress_keys(cfg: WorkloadConfig, layer: int, frame: int) -> np.ndarray:
    """i.i.d. keys, then per (frame, kv head): 2% of tokens scaled x4, 10% copy one of 32 template rows."""
    H, T, d = cfg.n_kv_heads, cfg.tokens_per_frame, cfg.head_dim
    k = iid(stream_key(cfg.seed, layer, frame, TENSOR_K), (H, T, d), "bf16").copy()
    tmpl = iid(stream_key(cfg.seed, layer, 0, TENSOR_STRESS_TMPL), (H, STRESS_TEMPLATES, d), "bf16")
    rank = raw_bits(stream_key(cfg.seed, layer, frame, TENSOR_STRESS_RANK), H * T).reshape(H, T)
    pick = raw_bits(stream_key(cfg.seed, layer, frame, TENSOR_STRESS_PICK), H * T).reshape(H, T)
    n_heavy = int(round(STRESS_HEAVY_FRACTION * T))
    n_dup = int(round(STRESS_DUP_FRACTION * T))
    for g in range(H):
        order = np.argsort(rank[g], kind="stable")
        for t in order[n_heavy:n_heavy + n_dup]:
            k[g, t] = tmpl[g, int(pick[g, t] % np.uint64(STRESS_TEMPLATES))]
        heavy = order[:n_heavy]
        k[g, heavy] = f32_to_bf16_bits(bf16_to_f32(k[g, heavy]) * np.float32(STRESS_HEAVY_MULT))
    return k


def frame_inputs(cfg: WorkloadConfig, layer: int, frame: int) -> dict:
    """Q [H_q, T, d], K and V [H_kv, T, d] of one layer and frame, in storage form
    (uint16 bf16 bit patterns, or float32)."""
    Hq, Hkv, T, d, dt = cfg.n_q_heads, cfg.n_kv_heads, cfg.tokens_per_frame, cfg.head_dim, cfg.dtype
    q = iid(stream_key(cfg.seed, layer, frame, TENSOR_Q), (Hq, T, d), dt)
    v = iid(stream_key(cfg.seed, layer, frame, TENSOR_V), (Hkv, T, d), dt)
    if cfg.recipe == "iid":
        k = iid(stream_key(cfg.seed, layer, frame, TENSOR_K), (Hkv, T, d), dt)
    elif cfg.recipe == "lowrank":
        k = _lowrank_keys(cfg, layer, frame)
    elif cfg.recipe == "stress":
        k = _stress_keys(cfg, layer, frame)
    else:
        raise ValueError(cfg.recipe)
    return {"q": q, "k": k, "v": v}


def frame_inputs_f64(cfg: WorkloadConfig, layer: int, frame: int) -> dict:
    raw = frame_inputs(cfg, layer, frame)
    return {n: to_f64(a, cfg.dtype) for n, a in raw.items()}
