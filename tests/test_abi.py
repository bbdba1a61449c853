"""Host-side checks of the C ABI: no GPU needed, no compute calls.

* the built library loads and exports every function declared in include/statekv.h;
* the ctypes mirrors of the public structs match the C layout (offsets from a
  small C program compiled with gcc against the header);
* argument validation happens before any HIP call and returns the documented
  statuses.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2605_31598_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "statekv.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(skv_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libstatekv.so is not built: run python paper_2605_31598_amd/build.py")
    return B.load_library()


def test_library_exports_every_declared_symbol(lib):
    declared = header_functions()
    assert set(declared) == set(B.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r" T (skv_[a-z_]+)$", out, flags=re.M))
    missing = [s for s in declared if s not in exported]
    assert not missing, f"declared but not exported: {missing}"
    for s in declared:
        getattr(lib, s)


def test_struct_layouts_match_header(tmp_path):
    prog = tmp_path / "layout.c"
    prog.write_text(r'''
#include <stddef.h>
#include <stdio.h>
#include "statekv.h"
#define F(T, m) printf(#T "." #m " %zu\n", offsetof(T, m));
int main(void) {
  F(skv_config, n_layers) F(skv_config, n_q_heads) F(skv_config, n_kv_heads) F(skv_config, head_dim)
  F(skv_config, tokens_per_frame) F(skv_config, capacity) F(skv_config, max_frames) F(skv_config, dtype)
  F(skv_config, softmax_scale) F(skv_config, pos_offset) F(skv_config, policy) F(skv_config, max_decode_tokens)
  F(skv_config, rope) F(skv_config, rope_theta) F(skv_config, rope_factor) F(skv_config, rope_orig_max)
  F(skv_config, split_refresh) F(skv_config, key_split_mode)
  F(skv_state_view_t, k) F(skv_state_view_t, v) F(skv_state_view_t, pos) F(skv_state_view_t, score)
  F(skv_state_view_t, size) F(skv_state_view_t, capacity) F(skv_state_view_t, frame)
  F(skv_state_view_t, pool_score) F(skv_state_view_t, pool_pos) F(skv_state_view_t, pool_size)
  F(skv_state_view_t, pool_stride)
  F(skv_cache_view_t, k) F(skv_cache_view_t, v) F(skv_cache_view_t, n_tokens) F(skv_cache_view_t, max_tokens)
  F(skv_cache_view_t, n_kv_heads) F(skv_cache_view_t, head_dim) F(skv_cache_view_t, decode_row0)
  F(skv_cache_view_t, decode_tokens)
  printf("sizeof.skv_config %zu\nsizeof.skv_state_view_t %zu\nsizeof.skv_cache_view_t %zu\n",
         sizeof(skv_config), sizeof(skv_state_view_t), sizeof(skv_cache_view_t));
  return 0;
}
''')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), str(prog), "-o", str(exe)], check=True)
    lines = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = dict(l.split() for l in lines if l.strip())
    for cls in (B.skv_config, B.skv_state_view_t, B.skv_cache_view_t):
        for name, _ in cls._fields_:
            assert int(got[f"{cls.__name__}.{name}"]) == getattr(cls, name).offset, (cls.__name__, name)
        assert int(got[f"sizeof.{cls.__name__}"]) == ctypes.sizeof(cls)


def _cfg(**kw):
    base = dict(n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=128, tokens_per_frame=16, capacity=32,
                max_frames=4, dtype=B.SKV_BF16, softmax_scale=0.0, pos_offset=0)
    base.update(kw)
    return B.skv_config(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(n_layers=0), B.SKV_ERR_INVALID_ARG),
    (dict(n_q_heads=6, n_kv_heads=4), B.SKV_ERR_INVALID_ARG),
    (dict(head_dim=96), B.SKV_ERR_UNSUPPORTED),
    (dict(capacity=-1), B.SKV_ERR_INVALID_ARG),
    (dict(tokens_per_frame=0), B.SKV_ERR_INVALID_ARG),
    (dict(max_frames=0), B.SKV_ERR_INVALID_ARG),
    (dict(dtype=7), B.SKV_ERR_INVALID_ARG),
    (dict(softmax_scale=-1.0), B.SKV_ERR_INVALID_ARG),
    (dict(softmax_scale=float("nan")), B.SKV_ERR_INVALID_ARG),
    (dict(capacity=16000, tokens_per_frame=729), B.SKV_ERR_UNSUPPORTED),
    (dict(max_frames=2 ** 30, tokens_per_frame=4), B.SKV_ERR_INVALID_ARG),
    (dict(pos_offset=-3), B.SKV_ERR_INVALID_ARG),
    (dict(policy=3), B.SKV_ERR_INVALID_ARG),
    (dict(policy=-1), B.SKV_ERR_INVALID_ARG),
    (dict(max_decode_tokens=-1), B.SKV_ERR_INVALID_ARG),
    (dict(rope=3, rope_theta=1e4), B.SKV_ERR_INVALID_ARG),
    (dict(rope=1, rope_theta=0.0), B.SKV_ERR_INVALID_ARG),
    (dict(rope=2, rope_theta=1e4, rope_factor=0.5, rope_orig_max=4096), B.SKV_ERR_INVALID_ARG),
    (dict(rope=2, rope_theta=1e4, rope_factor=4.0, rope_orig_max=0), B.SKV_ERR_INVALID_ARG),
    (dict(split_refresh=2), B.SKV_ERR_INVALID_ARG),
    (dict(key_split_mode=3), B.SKV_ERR_INVALID_ARG),
    (dict(key_split_mode=-1), B.SKV_ERR_INVALID_ARG),
])
def test_init_rejects_bad_configs_before_touching_the_device(lib, kw, status):
    h = ctypes.c_void_p(123)
    cfg = _cfg(**kw)
    assert lib.skv_init(ctypes.byref(cfg), None, ctypes.byref(h)) == status
    assert h.value is None
    assert lib.skv_last_error()


def test_null_arguments(lib):
    h = ctypes.c_void_p()
    assert lib.skv_init(None, None, ctypes.byref(h)) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_init(ctypes.byref(_cfg()), None, None) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_frame_step(None, 0, 1, None, None, None, None) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_decode_step(None, 0, 1, 1, None, None, None, None) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_state_view(None, 0, None) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_decode_cache_view(None, 0, None) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_reset(None) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_seek(None, 0) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_timing_start(None, 4) == B.SKV_ERR_INVALID_ARG
    assert lib.skv_timing_stride(None, 8) == B.SKV_ERR_INVALID_ARG
    lib.skv_destroy(None)


def test_stage_enum_matches_binding():
    text = open(HEADER).read()
    for i, name in enumerate(("SKV_STAGE_ATTENTION", "SKV_STAGE_REFRESH", "SKV_STAGE_STATE_UPDATE", "SKV_STAGE_APPEND",
                              "SKV_N_STAGES")):
        assert f"{name} = {i}" in text
    assert B.N_STAGES == 4 and len(B.STAGES) == 4


def test_status_strings(lib):
    for s, name in [(0, "SKV_OK"), (-1, "SKV_ERR_INVALID_ARG"), (-2, "SKV_ERR_OUT_OF_MEMORY"),
                    (-3, "SKV_ERR_CAPACITY"), (-4, "SKV_ERR_ORDER"), (-5, "SKV_ERR_DEVICE"),
                    (-6, "SKV_ERR_UNSUPPORTED")]:
        assert B.status_string(s) == name


def test_product_path_fails_loudly_without_library(tmp_path):
    saved = B._lib
    try:
        B._lib = None
        with pytest.raises(RuntimeError, match="missing"):
            B.load_library(str(tmp_path / "nope.so"))
    finally:
        B._lib = saved
