"""Seeded input generator: published test vectors, determinism and the recipes' structure."""
import numpy as np

from workloads import CONFIGS, generate as gen
from workloads.configs import ORDER


def test_splitmix64_published_sequence():
    # SplitMix64 seeded with 0 (Steele, Lea & Flood 2014): the first four outputs.
    expect = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC]
    assert [gen.mix64_int(i * gen.GOLDEN) for i in range(1, 5)] == expect
    np.testing.assert_array_equal(gen.raw_bits(0, 4), np.array(expect, dtype=np.uint64))


def test_vectorised_and_scalar_hash_agree():
    key = gen.stream_key(123, 4, 9, gen.TENSOR_Q)
    bits = gen.raw_bits(key, 100, start=17)
    for i in range(100):
        assert int(bits[i]) == gen.mix64_int(key + (17 + i + 1) * gen.GOLDEN)


def test_normal_table_moments_and_symmetry():
    t = gen.normal_table("f32").astype(np.float64)
    assert abs(t.mean()) < 1e-6 and abs(t.std() - 1.0) < 2e-3
    np.testing.assert_array_equal(t, -t[::-1])
    tb = gen.bf16_to_f64(gen.normal_table("bf16"))
    assert np.max(np.abs(tb - t) / np.maximum(np.abs(t), 1e-30)) <= 2.0 ** -8


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 3.0e38], dtype=np.float32)
    got = gen.bf16_to_f32(gen.f32_to_bf16_bits(x))
    np.testing.assert_array_equal(got, np.array([1.0, 1.0, 1.0 + 4 * 2 ** -8, 1.0, -2.5, got[5]], dtype=np.float32))
    assert abs(got[5] - 3.0e38) / 3.0e38 < 2 ** -8


def test_frames_are_deterministic_and_distinct():
    cfg = CONFIGS["vlm7b_1layer"]
    a = gen.frame_inputs(cfg, 0, 3)
    b = gen.frame_inputs(cfg, 0, 3)
    c = gen.frame_inputs(cfg, 0, 4)
    for n in ("q", "k", "v"):
        np.testing.assert_array_equal(a[n], b[n])
        assert not np.array_equal(a[n], c[n])
        assert a[n].dtype == np.uint16
    assert a["q"].shape == (28, 196, 128) and a["k"].shape == (4, 196, 128)
    x = gen.bf16_to_f64(a["q"])
    assert abs(x.mean()) < 0.01 and abs(x.std() - 1) < 0.01


def test_tiny_is_fp32():
    x = gen.frame_inputs(CONFIGS["tiny_f32"], 0, 0)
    assert x["q"].dtype == np.float32 and x["q"].shape == (4, 16, 64)


def test_lowrank_keys_share_a_component_across_frames():
    cfg = CONFIGS["vlm72b_80layer"]
    k0 = gen.bf16_to_f64(gen.frame_inputs(cfg, 5, 0)["k"])
    k1 = gen.bf16_to_f64(gen.frame_inputs(cfg, 5, 1)["k"])
    assert k0.shape == (8, 256, 128)
    # variance of c.W/4 is 16/16 = 1, noise 0.25 -> per-element variance about 1.25
    assert abs(k0.var() - 1.25) < 0.1
    # keys of one KV head live near a 16-dimensional subspace shared by all frames
    g = 2
    basis = np.linalg.svd(k0[g], full_matrices=False)[2][:16]
    resid = k1[g] - (k1[g] @ basis.T) @ basis
    assert resid.var() < 0.35


def test_stress_keys_have_heavy_rows_and_exact_duplicates():
    cfg = CONFIGS["stress_1layer"]
    k = gen.frame_inputs(cfg, 0, 7)["k"]
    k2 = gen.frame_inputs(cfg, 0, 8)["k"]
    assert k.shape == (8, 729, 128)
    norms = np.linalg.norm(gen.bf16_to_f64(k), axis=2)
    for g in range(8):
        assert int((norms[g] > 2.5 * np.median(norms[g])).sum()) == 15
        rows = {r.tobytes() for r in k[g]}
        assert len(rows) <= 729 - 73 + 32  # 73 copies of at most 32 templates
        # templates recur in the next frame: exact duplicates across frames
        assert len(rows & {r.tobytes() for r in k2[g]}) > 0


def test_config_registry_shapes():
    assert ORDER == list(CONFIGS)
    c3 = CONFIGS["vlm7b_28layer"]
    assert (c3.n_layers, c3.group, c3.capacity, c3.full_from_frame) == (28, 7, 2048, 11)
    assert CONFIGS["vlm72b_80layer"].full_from_frame == 16
    assert CONFIGS["stress_1layer"].full_from_frame == 12
    assert CONFIGS["tiny_f32"].state_size(1) == 16 and CONFIGS["tiny_f32"].state_size(5) == 32
