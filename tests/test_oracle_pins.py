"""Pins of the fp64 CPU oracle against things other than itself.

* a hand-derived worked example with rational answers (tests/golden);
* a pure-Python brute force on tiny inputs;
* the library routine torch SDPA (causal, fp64, CPU): with capacity >= all tokens
  the streaming step is exact full causal self-attention, with capacity 0 it is
  per-frame causal attention; SDPA with one-hot values returns the attention
  matrix itself, which pins the scores;
* closed forms at Q = 0 (uniform attention) including the lowest-position tie rule;
* invariants: rows of A sum to 1, scores of a KV head sum to G, state size is
  min(B, seen), per-frame work is constant once the state is full, state order
  does not matter.

The planted-mistake test at the end swaps one oracle step for a plausible wrong
variant and checks that some pin fails.
"""
from __future__ import annotations

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import bruteforce as bf
from oracle import statekv_oracle as orc

HERE = os.path.dirname(os.path.abspath(__file__))


# ----------------------------------------------------------------------------
# helpers
# ----------------------------------------------------------------------------
def random_video(seed, H_q, H_kv, d, T, N, kscale=1.0):
    rng = np.random.default_rng(seed)
    return [
        (rng.standard_normal((H_q, T, d)), kscale * rng.standard_normal((H_kv, T, d)),
         rng.standard_normal((H_kv, T, d)))
        for _ in range(N)
    ]


def run_oracle(video, B, scale=None, pos_offset=0, keep_attn=False):
    H_kv, _, d = video[0][1].shape
    st = orc.LayerState.empty(H_kv, d)
    res = []
    for n, (q, k, v) in enumerate(video):
        r = orc.frame_step(st, q, k, v, n, B, scale, pos_offset, keep_attn=keep_attn)
        st = r.state
        res.append(r)
    return res


def sdpa_causal(q, k, v, scale):
    """torch SDPA, causal, fp64 on CPU; GQA by repeating each KV head G times (contiguous groups)."""
    G = q.shape[0] // k.shape[0]
    kt = torch.from_numpy(k).repeat_interleave(G, dim=0)
    vt = torch.from_numpy(v).repeat_interleave(G, dim=0)
    o = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], kt[None], vt[None], is_causal=True, scale=scale)
    return o[0].numpy()


def _val(x):
    if isinstance(x, str) and x.startswith("ln"):
        return math.log(int(x[2:]))
    return float(x)


def _frac(x):
    return float(Fraction(x))


# ----------------------------------------------------------------------------
# pin checks (raise AssertionError; reused by the planted-mistake test)
# ----------------------------------------------------------------------------
def check_golden():
    with open(os.path.join(HERE, "golden", "handworked_three_frames.json")) as f:
        gold = json.load(f)
    c = gold["config"]
    st = orc.LayerState.empty(c["n_kv_heads"], c["head_dim"])
    for n, fr in enumerate(gold["frames"]):
        q = np.vectorize(_val, otypes=[float])(np.array(fr["q"], dtype=object))
        k = np.array(fr["k"], dtype=float)
        v = np.array(fr["v"], dtype=float)
        r = orc.frame_step(st, q, k, v, n, c["capacity"], c["scale"], c["pos_offset"])
        exp_out = np.vectorize(_frac, otypes=[float])(np.array(fr["expect_out"], dtype=object))
        exp_s = np.vectorize(_frac, otypes=[float])(np.array(fr["expect_scores"], dtype=object))
        np.testing.assert_allclose(r.out, exp_out, rtol=0, atol=1e-12)
        np.testing.assert_array_equal(r.pool_pos, np.array(fr["expect_pool_pos"]))
        np.testing.assert_allclose(r.pool_score, exp_s, rtol=0, atol=1e-12)
        np.testing.assert_array_equal(r.state.pos, np.array(fr["expect_state_pos"]))
        st = r.state


def check_full_capacity_is_causal_sdpa(seed=1, H_q=6, H_kv=2, d=8, T=5, N=4):
    video = random_video(seed, H_q, H_kv, d, T, N)
    scale = d ** -0.5
    res = run_oracle(video, B=N * T, scale=scale)
    q = np.concatenate([x[0] for x in video], axis=1)
    k = np.concatenate([x[1] for x in video], axis=1)
    v = np.concatenate([x[2] for x in video], axis=1)
    o_full = sdpa_causal(q, k, v, scale)
    L = N * T
    # one-hot values make SDPA return the attention matrix itself
    A_full = sdpa_causal(q, k, np.broadcast_to(np.eye(L), (H_kv, L, L)).copy(), scale)
    G = H_q // H_kv
    for n, r in enumerate(res):
        rows = slice(n * T, (n + 1) * T)
        np.testing.assert_allclose(r.out, o_full[:, rows], rtol=0, atol=1e-12)
        # pool = every earlier token (state, ascending position) then the frame
        assert np.array_equal(r.pool_pos[0], np.arange((n + 1) * T))
        s_ref = A_full[:, rows, : (n + 1) * T].reshape(H_kv, G, T, -1).sum(axis=(1, 2)) / T
        np.testing.assert_allclose(r.pool_score, s_ref, rtol=0, atol=1e-12)


def check_zero_capacity_is_framewise_sdpa(seed=2, H_q=4, H_kv=2, d=8, T=6, N=3):
    video = random_video(seed, H_q, H_kv, d, T, N)
    scale = d ** -0.5
    res = run_oracle(video, B=0, scale=scale)
    for r, (q, k, v) in zip(res, video):
        np.testing.assert_allclose(r.out, sdpa_causal(q, k, v, scale), rtol=0, atol=1e-12)
        assert r.state.size == 0


def check_full_policy_is_causal_sdpa(seed=5, H_q=6, H_kv=3, d=8, T=4, N=5, B=3):
    """Full SA: whatever the capacity, frame n attends to every earlier token, so the
    outputs of the stream are one causal attention over all N*T tokens."""
    video = random_video(seed, H_q, H_kv, d, T, N)
    scale = d ** -0.5
    st = orc.LayerState.empty(H_kv, d)
    q = np.concatenate([x[0] for x in video], axis=1)
    k = np.concatenate([x[1] for x in video], axis=1)
    v = np.concatenate([x[2] for x in video], axis=1)
    o_full = sdpa_causal(q, k, v, scale)
    for n, (qn, kn, vn) in enumerate(video):
        r = orc.frame_step(st, qn, kn, vn, n, B, scale, policy="full")
        np.testing.assert_allclose(r.out, o_full[:, n * T:(n + 1) * T], rtol=0, atol=1e-12)
        assert np.array_equal(r.state.pos, np.tile(np.arange((n + 1) * T), (H_kv, 1)))
        st = r.state


def check_recent_policy_window(seed=6, H_q=4, H_kv=2, d=8, T=5, N=6, B=7, pos_offset=3):
    """Recency window: the state entering frame n is the last min(B, n*T) tokens, and the
    frame attends to exactly those (fully visible) plus itself (causal)."""
    video = random_video(seed, H_q, H_kv, d, T, N)
    scale = d ** -0.5
    st = orc.LayerState.empty(H_kv, d)
    ks = np.concatenate([x[1] for x in video], axis=1)
    vs = np.concatenate([x[2] for x in video], axis=1)
    G = H_q // H_kv
    for n, (qn, kn, vn) in enumerate(video):
        S = min(B, n * T)
        np.testing.assert_array_equal(st.pos, np.tile(pos_offset + np.arange(n * T - S, n * T), (H_kv, 1)))
        r = orc.frame_step(st, qn, kn, vn, n, B, scale, pos_offset, policy="recent")
        keys = slice(n * T - S, (n + 1) * T)
        allow = np.zeros((T, S + T), dtype=bool)
        for i in range(T):
            allow[i, :S + i + 1] = True
        o = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(qn)[None], torch.from_numpy(ks[:, keys]).repeat_interleave(G, dim=0)[None],
            torch.from_numpy(vs[:, keys]).repeat_interleave(G, dim=0)[None],
            attn_mask=torch.from_numpy(allow), scale=scale)[0].numpy()
        np.testing.assert_allclose(r.out, o, rtol=0, atol=1e-12)
        st = r.state


def check_decode_is_causal_sdpa(seed=8, H_q=6, H_kv=2, d=8, T=4, N=3, chunks=(1, 3, 1)):
    """Decoding over D: after N frames, chunks of t new tokens; every decoded token's output
    equals one causal attention over the whole stream (video tokens, then decoded tokens)."""
    rng = np.random.default_rng(seed)
    n_dec = sum(chunks)
    L = N * T + n_dec
    q = rng.standard_normal((H_q, L, d))
    k = rng.standard_normal((H_kv, L, d))
    v = rng.standard_normal((H_kv, L, d))
    scale = d ** -0.5
    ref = sdpa_causal(q, k, v, scale)
    pos = N * T
    for t in chunks:
        new = slice(pos, pos + t)
        o = orc.decode_attention(q[:, new], k[:, :pos], v[:, :pos], k[:, new], v[:, new], scale)
        np.testing.assert_allclose(o, ref[:, new], rtol=0, atol=1e-12)
        pos += t


def check_rope_closed_form():
    """d = 4, theta = 100: pair frequencies 1 and 1/10; unit vectors rotate in the planes
    (0, 2) and (1, 3) by p and p/10, counter-clockwise, and keep their norm."""
    spec = orc.rope_spec(4, 100.0, dtype="f32")
    p = np.array([0.0, 1.0, 7.0, 1234.0])
    e0 = np.broadcast_to(np.array([1.0, 0.0, 0.0, 0.0]), (4, 4))
    e1 = np.broadcast_to(np.array([0.0, 1.0, 0.0, 0.0]), (4, 4))
    e3 = np.broadcast_to(np.array([0.0, 0.0, 0.0, 1.0]), (4, 4))
    np.testing.assert_allclose(orc.rope_rotate(e0, p, spec), np.stack([np.cos(p), 0 * p, np.sin(p), 0 * p], 1),
                               atol=1e-7)
    np.testing.assert_allclose(orc.rope_rotate(e1, p, spec),
                               np.stack([0 * p, np.cos(p / 10), 0 * p, np.sin(p / 10)], 1), atol=1e-7)
    np.testing.assert_allclose(orc.rope_rotate(e3, p, spec),
                               np.stack([0 * p, -np.sin(p / 10), 0 * p, np.cos(p / 10)], 1), atol=1e-7)


def check_rope_relative_positions(seed=10, H_q=4, H_kv=2, d=8, T=4, N=4, B=6):
    """RoPE logits depend only on position differences, so shifting the whole stream's
    virtual positions (pos_offset) changes neither outputs nor scores (fp32-rounded
    rotations: to rounding), while the stored positions shift."""
    video = random_video(seed, H_q, H_kv, d, T, N)
    spec = orc.rope_spec(d, 10000.0, dtype="f32")
    runs = []
    for off in (0, 100000):
        st = orc.LayerState.empty(H_kv, d)
        res = []
        for n, (q, k, v) in enumerate(video):
            r = orc.frame_step(st, q, k, v, n, B, d ** -0.5, off, rope=spec)
            st = r.state
            res.append(r)
        runs.append(res)
    for a, b in zip(*runs):
        np.testing.assert_allclose(a.out, b.out, atol=2e-5)
        np.testing.assert_allclose(a.pool_score, b.pool_score, rtol=1e-4)
        assert np.array_equal(a.pool_pos + 100000, b.pool_pos)


def check_yarn_limits():
    """YaRN with s = 1 is plain RoPE; with s > 1 the highest frequency (r >> 32) is kept,
    the lowest (r < 1) is divided by s, and cos/sin carry 0.1 ln(s) + 1."""
    plain = orc.rope_spec(128, 1e4)
    same = orc.rope_spec(128, 1e4, "yarn", factor=1.0, orig_max=4096)
    np.testing.assert_allclose(same.freqs, plain.freqs, rtol=1e-15, atol=0)
    assert same.mscale == 1.0
    y = orc.rope_spec(128, 1e4, "yarn", factor=8.0, orig_max=4096)
    assert y.freqs[0] == plain.freqs[0]
    np.testing.assert_allclose(y.freqs[-1], plain.freqs[-1] / 8.0, rtol=1e-15)
    assert abs(y.mscale - (0.1 * math.log(8.0) + 1.0)) < 1e-15
    assert np.all(np.diff(y.freqs) < 0) and np.all(y.freqs <= plain.freqs)


def check_zero_query_closed_form(H_q=6, H_kv=3, d=4, T=5, N=6, B=7):
    G = H_q // H_kv
    rng = np.random.default_rng(3)
    video = [(np.zeros((H_q, T, d)), rng.standard_normal((H_kv, T, d)),
              rng.standard_normal((H_kv, T, d))) for _ in range(N)]
    res = run_oracle(video, B)
    for n, r in enumerate(res):
        S = min(B, n * T)
        inv = [1.0 / (S + i + 1) for i in range(T)]
        s_state = G / T * sum(inv)
        s_frame = [G / T * sum(inv[t:]) for t in range(T)]
        expect = np.array([s_state] * S + s_frame)
        np.testing.assert_allclose(r.pool_score, np.broadcast_to(expect, (H_kv, S + T)), rtol=1e-13, atol=0)
        # uniform attention makes the earliest tokens win every tie: the state is the first B tokens
        keep = min(B, (n + 1) * T)
        np.testing.assert_array_equal(r.state.pos, np.broadcast_to(np.arange(keep), (H_kv, keep)))


def check_bruteforce(seed, H_q, H_kv, d, T, B, N, pos_offset):
    video = random_video(seed, H_q, H_kv, d, T, N, kscale=1.5)
    scale = 0.7
    res = run_oracle(video, B, scale=scale, pos_offset=pos_offset)
    state = [[] for _ in range(H_kv)]
    for n, ((q, k, v), r) in enumerate(zip(video, res)):
        b = bf.step(q.tolist(), state, k.tolist(), v.tolist(), n, B, scale, pos_offset)
        np.testing.assert_allclose(r.out, np.array(b["out"]), rtol=0, atol=1e-12)
        np.testing.assert_allclose(r.pool_score, np.array(b["scores"]), rtol=0, atol=1e-12)
        np.testing.assert_array_equal(r.pool_pos, np.array(b["pool_pos"]))
        for g in range(H_kv):
            np.testing.assert_array_equal(r.state.pos[g], [e[0] for e in b["new_state"][g]])
            np.testing.assert_array_equal(r.state.k[g].reshape(-1, d), np.array([e[1] for e in b["new_state"][g]]).reshape(-1, d))
        state = b["new_state"]


# ----------------------------------------------------------------------------
# tests
# ----------------------------------------------------------------------------
def test_full_policy_equals_causal_sdpa_over_the_stream():
    check_full_policy_is_causal_sdpa()


def test_recent_policy_keeps_the_last_tokens():
    check_recent_policy_window()
    check_recent_policy_window(seed=7, T=4, B=8, N=5, pos_offset=0)  # window of whole frames


def test_decode_over_the_detailed_cache_equals_causal_sdpa():
    check_decode_is_causal_sdpa()
    check_decode_is_causal_sdpa(seed=9, H_q=7, H_kv=1, d=16, T=5, N=2, chunks=(4, 2))


def test_rope_closed_form_and_relative_positions():
    check_rope_closed_form()
    check_rope_relative_positions()


def test_yarn_reduces_to_rope_and_blends_by_wavelength():
    check_yarn_limits()


def check_yarn_ramp_interior():
    """YaRN's ramp between its limits: two pairs whose wavelength ratio lies strictly inside
    (1, 32), against values worked by hand from YaRN's definition
    (tests/golden/yarn_ramp_interior.json holds the derivation)."""
    import json

    g = json.load(open(os.path.join(HERE, "golden", "yarn_ramp_interior.json")))
    c = g["config"]
    spec = orc.rope_spec(c["head_dim"], c["theta"], "yarn", factor=c["factor"], orig_max=c["orig_max"], dtype="f32")
    np.testing.assert_allclose(spec.freqs, g["expect_freqs"], rtol=1e-12)
    assert abs(spec.mscale - g["expect_mscale"]) <= 1e-12
    d, half, p = c["head_dim"], c["head_dim"] // 2, g["rotation_position"]
    for j, (cos_m, sin_m) in g["expect_rotated_unit"].items():
        j = int(j)
        x = np.zeros((1, d))
        x[0, j] = 1.0
        y = orc.rope_rotate(x, np.array([p]), spec)[0]
        np.testing.assert_allclose([y[j], y[j + half]], [cos_m, sin_m], rtol=2e-7)  # rounded to fp32
        others = np.delete(y, [j, j + half])
        assert np.all(others == 0.0)


def test_yarn_ramp_interior_hand_worked():
    check_yarn_ramp_interior()


def test_rope_bf16_rounding_matches_a_library_conversion():
    x = np.random.default_rng(3).standard_normal(4096) * 10.0 ** np.random.default_rng(4).uniform(-3, 3, 4096)
    ref = torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(orc.round_to_dtype(x, "bf16"), ref)


def test_golden_handworked():
    check_golden()


def test_full_capacity_equals_causal_sdpa():
    check_full_capacity_is_causal_sdpa()


def test_full_capacity_equals_causal_sdpa_gqa7():
    check_full_capacity_is_causal_sdpa(seed=11, H_q=14, H_kv=2, d=16, T=7, N=3)


def test_zero_capacity_equals_framewise_causal_sdpa():
    check_zero_capacity_is_framewise_sdpa()


def test_zero_query_closed_form_and_earliest_state():
    check_zero_query_closed_form()


@pytest.mark.parametrize("seed,H_q,H_kv,d,T,B,N,pos_offset", [
    (0, 2, 1, 3, 3, 4, 4, 0),
    (1, 4, 2, 4, 4, 3, 4, 5),   # B < T
    (2, 3, 3, 2, 5, 0, 3, 0),   # B = 0
    (3, 6, 2, 5, 2, 100, 4, 0),  # B larger than every pool
    (4, 4, 1, 3, 1, 2, 5, 7),   # T = 1
    (5, 6, 3, 4, 6, 8, 3, 0),   # B not a multiple of T
])
def test_vectorised_matches_bruteforce(seed, H_q, H_kv, d, T, B, N, pos_offset):
    check_bruteforce(seed, H_q, H_kv, d, T, B, N, pos_offset)


def test_attention_rows_sum_to_one_and_mask():
    video = random_video(4, 8, 2, 16, 9, 4)
    for n, r in enumerate(run_oracle(video, B=12, keep_attn=True)):
        S = min(12, n * 9)
        np.testing.assert_allclose(r.attn.sum(axis=2), 1.0, rtol=0, atol=1e-13)
        vis = orc.visibility(S, 9)
        assert np.all(r.attn[:, ~vis] == 0.0)
        assert np.all(r.attn[:, vis] > 0.0)


def test_scores_of_a_kv_head_sum_to_group_size():
    video = random_video(5, 12, 3, 8, 6, 5)
    for r in run_oracle(video, B=10):
        np.testing.assert_allclose(r.pool_score.sum(axis=1), 4.0, rtol=0, atol=1e-12)
        assert np.all(r.pool_score > 0)  # every key is visible to the frame's last query


@pytest.mark.parametrize("T,B", [(5, 12), (4, 8), (6, 3), (3, 0)])
def test_state_size_is_min_capacity_seen(T, B):
    video = random_video(6, 4, 2, 4, T, 6)
    for n, r in enumerate(run_oracle(video, B)):
        assert r.state.size == min(B, (n + 1) * T)
        assert r.pool_pos.shape[1] == min(B, n * T) + T
        assert np.all(np.diff(r.state.pos, axis=1) > 0)  # canonical ascending order, no repeats


def test_per_frame_work_constant_once_full():
    H_q, H_kv, d, T, B, N = 4, 2, 8, 5, 12, 8
    res = run_oracle(random_video(7, H_q, H_kv, d, T, N), B)
    flops = [r.flops for r in res]
    full = -(-B // T)
    for n, f in enumerate(flops):
        assert f == orc.attention_flops(H_q, d, T, min(B, n * T))
    assert len(set(flops[full:])) == 1
    assert all(flops[n] < flops[n + 1] for n in range(full))


def test_state_order_does_not_matter():
    rng = np.random.default_rng(8)
    H_q, H_kv, d, T, S = 6, 2, 8, 4, 9
    st = orc.LayerState(pos=np.tile(np.arange(S) * 3, (H_kv, 1)), k=rng.standard_normal((H_kv, S, d)),
                        v=rng.standard_normal((H_kv, S, d)), score=np.zeros((H_kv, S)))
    q, k, v = rng.standard_normal((H_q, T, d)), rng.standard_normal((H_kv, T, d)), rng.standard_normal((H_kv, T, d))
    perm = rng.permutation(S)
    st2 = orc.LayerState(st.pos[:, perm], st.k[:, perm], st.v[:, perm], st.score[:, perm])
    a = orc.frame_step(st, q, k, v, 10, 7)
    b = orc.frame_step(st2, q, k, v, 10, 7)
    np.testing.assert_allclose(a.out, b.out, rtol=0, atol=1e-13)
    np.testing.assert_allclose(a.pool_score[:, :S][:, perm], b.pool_score[:, :S], rtol=0, atol=1e-13)
    np.testing.assert_array_equal(a.state.pos, b.state.pos)


def test_duplicate_keys_tie_exactly_and_lower_position_wins():
    rng = np.random.default_rng(9)
    H_q, H_kv, d, T, S = 4, 1, 8, 3, 5
    row = rng.standard_normal(d)
    # all state keys identical -> bit-identical scores; frame keys point away from the queries
    st = orc.LayerState(pos=np.array([[2, 5, 11, 17, 23]]), k=np.tile(row, (1, S, 1)),
                        v=rng.standard_normal((1, S, d)), score=np.zeros((1, S)))
    q = np.abs(rng.standard_normal((H_q, T, d))) * np.sign(row)
    k = -4.0 * np.abs(rng.standard_normal((1, T, d))) * np.sign(row)
    r = orc.frame_step(st, q, k, rng.standard_normal((1, T, d)), 30, 3)
    s = r.pool_score[0]
    assert np.all(s[:S] == s[0])  # exact equality, not approximate
    assert np.all(s[S:] < s[0])
    np.testing.assert_array_equal(r.state.pos[0], [2, 5, 11])


def test_selection_against_full_sort_with_ties():
    rng = np.random.default_rng(10)
    for trial in range(50):
        P = int(rng.integers(1, 60))
        B = int(rng.integers(0, 70))
        s = rng.integers(0, 6, size=P) / 7.0  # many exact ties
        pos = rng.permutation(1000)[:P]
        got = orc.select_top(s, pos, B)
        ref = sorted(range(P), key=lambda j: (-s[j], pos[j]))[:min(B, P)]
        assert sorted(pos[got].tolist()) == sorted(pos[ref].tolist())
        assert np.all(np.diff(pos[got]) > 0)


def test_state_rows_are_input_bytes():
    video = random_video(12, 4, 2, 8, 5, 5)
    res = run_oracle(video, B=7)
    rows = {}
    for n, (q, k, v) in enumerate(video):
        for g in range(2):
            for t in range(5):
                rows[(g, n * 5 + t)] = (k[g, t], v[g, t])
    for r in res:
        for g in range(2):
            for j, p in enumerate(r.state.pos[g]):
                assert np.array_equal(r.state.k[g, j], rows[(g, int(p))][0])
                assert np.array_equal(r.state.v[g, j], rows[(g, int(p))][1])


def test_decode_cache_holds_every_frame_in_order():
    video = random_video(13, 4, 2, 8, 5, 4)
    inputs = lambda n: video[n]
    st, cache, res = orc.run_layer(inputs, 4, 6, 2, 8)
    K, V = cache.as_arrays()
    assert cache.n_tokens == 20
    np.testing.assert_array_equal(K, np.concatenate([x[1] for x in video], axis=1))
    np.testing.assert_array_equal(V, np.concatenate([x[2] for x in video], axis=1))
    assert st.size == 6


# ----------------------------------------------------------------------------
# planted mistakes: each plausible wrong variant of an oracle step fails a pin
# ----------------------------------------------------------------------------
def _mut_mask_strict(S, T):
    i = np.arange(T)[:, None]
    j = np.arange(S + T)[None, :]
    return (j < S) | ((j - S) < i) | ((j - S) == 0)


def _mut_mask_no_causal(S, T):
    return np.ones((T, S + T), dtype=bool)


def _mut_gqa_interleaved(H_q, H_kv):
    return np.arange(H_q) % H_kv


def _mut_scores_no_norm(A, n_kv_heads):
    H_q, T, P = A.shape
    return A.reshape(n_kv_heads, H_q // n_kv_heads, T, P).sum(axis=(1, 2))


def _mut_scores_mean_heads(A, n_kv_heads):
    H_q, T, P = A.shape
    return A.reshape(n_kv_heads, H_q // n_kv_heads, T, P).mean(axis=1).sum(axis=1) / T


def _mut_select_high_pos(scores, pos, capacity):
    P = scores.shape[0]
    keep = np.arange(P) if P <= capacity else np.lexsort((-pos, -scores))[:capacity]
    return keep[np.argsort(pos[keep], kind="stable")]


def _mut_select_lowest(scores, pos, capacity):
    P = scores.shape[0]
    keep = np.arange(P) if P <= capacity else np.lexsort((pos, scores))[:capacity]
    return keep[np.argsort(pos[keep], kind="stable")]


def _mut_positions_physical(frame, T, pos_offset=0):
    return pos_offset + np.arange(T, dtype=np.int64) + frame  # wrong: not from the virtual length


def _mut_rope_interleaved(x, positions, spec):
    ang = np.asarray(positions, dtype=np.float64)[:, None] * spec.freqs[None, :]
    c, s_ = np.cos(ang) * spec.mscale, np.sin(ang) * spec.mscale
    ev, od = x[..., 0::2], x[..., 1::2]  # wrong: adjacent pairs instead of (j, j + d/2)
    out = np.empty_like(x)
    out[..., 0::2] = ev * c - od * s_
    out[..., 1::2] = od * c + ev * s_
    return orc.round_to_dtype(out, spec.dtype)


_ROPE = orc.rope_rotate


def _mut_rope_clockwise(x, positions, spec):
    return _ROPE(x, -np.asarray(positions, dtype=np.float64), spec)  # wrong direction


_SPEC = orc.rope_spec


def _yarn_variant(head_dim, theta, kind, factor, orig_max, dtype, beta=32.0, invert=False, temperature=True):
    if kind != "yarn":
        return _SPEC(head_dim, theta, kind, factor, orig_max, dtype)
    j = np.arange(head_dim // 2, dtype=np.float64)
    f = theta ** (-2.0 * j / head_dim)
    g = np.clip((orig_max * f / (2.0 * np.pi) - 1.0) / (beta - 1.0), 0.0, 1.0)
    if invert:
        g = 1.0 - g
    return orc.RopeSpec((1.0 - g) * f / factor + g * f, 0.1 * np.log(factor) + 1.0 if temperature else 1.0, dtype)


def _mut_yarn_beta(head_dim, theta, kind="plain", factor=1.0, orig_max=0, dtype="bf16"):
    return _yarn_variant(head_dim, theta, kind, factor, orig_max, dtype, beta=64.0)  # wrong ramp edge


def _mut_yarn_inverted(head_dim, theta, kind="plain", factor=1.0, orig_max=0, dtype="bf16"):
    return _yarn_variant(head_dim, theta, kind, factor, orig_max, dtype, invert=True)  # interpolates the wrong end


def _mut_yarn_no_temperature(head_dim, theta, kind="plain", factor=1.0, orig_max=0, dtype="bf16"):
    return _yarn_variant(head_dim, theta, kind, factor, orig_max, dtype, temperature=False)


def _mut_recent_oldest(pos, capacity):
    P = pos.shape[0]
    keep = np.arange(P) if P <= capacity else np.argsort(pos, kind="stable")[:capacity]  # wrong: oldest
    return keep[np.argsort(pos[keep], kind="stable")]


PINS = [check_golden, check_full_capacity_is_causal_sdpa,
        lambda: check_full_capacity_is_causal_sdpa(seed=11, H_q=14, H_kv=2, d=16, T=7, N=3),
        check_zero_capacity_is_framewise_sdpa, check_zero_query_closed_form,
        lambda: check_bruteforce(1, 4, 2, 4, 4, 3, 4, 5), check_full_policy_is_causal_sdpa,
        check_recent_policy_window, check_decode_is_causal_sdpa, check_rope_closed_form,
        check_rope_relative_positions, check_yarn_limits, check_yarn_ramp_interior]


@pytest.mark.parametrize("name,attr,mutant", [
    ("mask off by one", "visibility", _mut_mask_strict),
    ("mask not causal", "visibility", _mut_mask_no_causal),
    ("GQA interleaved", "kv_head_of", _mut_gqa_interleaved),
    ("scores missing 1/T", "importance_scores", _mut_scores_no_norm),
    ("scores averaged over heads", "importance_scores", _mut_scores_mean_heads),
    ("ties to higher position", "select_top", _mut_select_high_pos),
    ("keeps the lowest scores", "select_top", _mut_select_lowest),
    ("positions from physical length", "frame_positions", _mut_positions_physical),
    ("recency window keeps the oldest", "select_recent", _mut_recent_oldest),
    ("RoPE pairs adjacent dimensions", "rope_rotate", _mut_rope_interleaved),
    ("RoPE rotates clockwise", "rope_rotate", _mut_rope_clockwise),
    ("YaRN ramp upper edge 64", "rope_spec", _mut_yarn_beta),
    ("YaRN ramp inverted", "rope_spec", _mut_yarn_inverted),
    ("YaRN without temperature", "rope_spec", _mut_yarn_no_temperature),
])
def test_planted_mistake_is_caught(monkeypatch, name, attr, mutant):
    monkeypatch.setattr(orc, attr, mutant)
    failed = 0
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed += 1
    assert failed > 0, f"no pin caught the planted mistake: {name}"
