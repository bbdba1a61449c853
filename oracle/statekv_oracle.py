"""Plain fp64 CPU oracle of StateKV's per-frame streaming video-prefill step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The GPU library never
calls it, and it shares no code with the GPU library.

Paper: "Linear Scaling Video VLMs for Long Video Understanding" (StateKV).
What one frame step computes, per layer and per KV head, in the paper's order
(Method, "Per-frame cache-builder forward pass"):

1. Candidate keys are the compressed state C_{n-1} (the only cross-frame
   context, Eq. 4) followed by the T tokens of frame n.
2. Attention of the frame's queries over [K_state; K_frame] with scale 1/sqrt(d_h)
   and mask M_n: state keys precede the frame, so they are always visible, and
   frame key t is visible to frame query i iff t <= i (Eq. 5).  Grouped-query
   attention maps query head h to KV head floor(h / G) (contiguous groups).
3. Importance of each candidate j: s_j = (1/T) * sum over the frame's queries of
   the normalised attention A_{i,j} (the score instantiation after the
   candidate-pool definition), aggregated by summing over the G query heads that
   share the KV head, because pruning is per layer and per KV head (Appendix A,
   shared protocol).
4. New state = the B candidates with the largest scores (Eq. 6); ties go to
   the lowest original token position; if the pool has <= B candidates all are
   kept.  Kept K/V rows are the input bytes, unchanged.
5. The frame's K/V rows are appended unchanged to the detailed decode cache
   D (never read during prefill), and the virtual length L_n grows by T;
   token positions come from L_n (virtual sequence length paragraph).

Two baselines of the evaluation share these steps and differ only in which
candidates survive step 4: the recency window (keep the B most recent
candidates, ReKV-style: the last B / T frames when T divides B) and streaming
full self-attention (Full SA: keep every candidate, so frame n attends to all
earlier tokens).

All arithmetic is fp64 NumPy.  Inputs are the exact bf16/fp32 values widened
to fp64.  Readings of points the paper leaves open are listed in the design
notes shipped with the repository and restated at each function below.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


# ----------------------------------------------------------------------------
# State
# ----------------------------------------------------------------------------
@dataclass
class LayerState:
    """Compressed state C of one layer: per KV head, S entries in ascending position.

    ``pos`` [H_kv, S] int64, ``k``/``v`` [H_kv, S, d] float64, ``score`` [H_kv, S]
    (score each entry had at the frame that last selected it; informational).
    """

    pos: np.ndarray
    k: np.ndarray
    v: np.ndarray
    score: np.ndarray

    @property
    def size(self) -> int:
        return int(self.pos.shape[1])

    @staticmethod
    def empty(n_kv_heads: int, head_dim: int) -> "LayerState":
        return LayerState(
            pos=np.zeros((n_kv_heads, 0), dtype=np.int64),
            k=np.zeros((n_kv_heads, 0, head_dim)),
            v=np.zeros((n_kv_heads, 0, head_dim)),
            score=np.zeros((n_kv_heads, 0)),
        )

    def copy(self) -> "LayerState":
        return LayerState(self.pos.copy(), self.k.copy(), self.v.copy(), self.score.copy())


@dataclass
class StepResult:
    out: np.ndarray  # [H_q, T, d] attention output (Eq. 5)
    attn: np.ndarray | None  # [H_q, T, S+T] normalised attention (kept only if asked)
    pool_pos: np.ndarray  # [H_kv, S+T] candidate positions (state entries, then frame tokens)
    pool_score: np.ndarray  # [H_kv, S+T] importance scores s_j
    kept: np.ndarray  # [H_kv, min(B, S+T)] indices into the pool, ascending position
    state: LayerState  # C_n
    flops: int  # multiply-add work of the attention, 4*d per visible (query, key) pair per head
    k_stored: np.ndarray | None = None  # the frame's keys as C and D store them (rotated with RoPE)


# ----------------------------------------------------------------------------
# Rotary position embedding at virtual positions
# ----------------------------------------------------------------------------
@dataclass
class RopeSpec:
    """RoPE applied to Q and K inside the step (virtual sequence length and RoPE scaling
    paragraphs): pair frequencies f_j (j < d/2), the cos/sin multiplier, and the dtype
    the rotated activations are rounded to ("bf16" or "f32", as the model stores them)."""

    freqs: np.ndarray
    mscale: float
    dtype: str


def rope_spec(head_dim, theta, kind="plain", factor=1.0, orig_max=0, dtype="bf16") -> RopeSpec:
    """f_j = theta^(-2j/d) (RoPE).  "yarn": YaRN's NTK-by-parts blend with scale s and original
    context L: r_j = L f_j / (2 pi), g_j = clamp((r_j - 1) / (32 - 1), 0, 1),
    f'_j = (1 - g_j) f_j / s + g_j f_j, and the temperature factor 0.1 ln(s) + 1 on cos/sin."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    f = theta ** (-2.0 * j / head_dim)
    if kind == "plain":
        return RopeSpec(f, 1.0, dtype)
    if kind != "yarn":
        raise ValueError(kind)
    r = orig_max * f / (2.0 * np.pi)
    g = np.clip((r - 1.0) / (32.0 - 1.0), 0.0, 1.0)
    return RopeSpec((1.0 - g) * f / factor + g * f, 0.1 * np.log(factor) + 1.0, dtype)


def round_to_dtype(x, dtype):
    """Round fp64 values to the nearest bf16 (ties to even) or fp32 value."""
    if dtype == "f32":
        return x.astype(np.float32).astype(np.float64)
    # bf16: nearest multiple of 2^(e-7) for x in [2^e, 2^(e+1)); ties to an even mantissa
    m, e = np.frexp(x)  # x = m 2^e, 0.5 <= |m| < 1
    scaled = np.ldexp(m, 8)  # 8 significant bits
    return np.ldexp(np.round(scaled), e - 8)  # np.round: half to even


def rope_rotate(x, positions, spec: RopeSpec):
    """x [..., P, d] at positions [P]: half-split pairs (j, j + d/2) rotated by p f_j, in fp64,
    then rounded to the spec's dtype."""
    h = x.shape[-1] // 2
    ang = np.asarray(positions, dtype=np.float64)[:, None] * spec.freqs[None, :]
    c = np.cos(ang) * spec.mscale
    s = np.sin(ang) * spec.mscale
    lo, hi = x[..., :h], x[..., h:]
    out = np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)
    return round_to_dtype(out, spec.dtype)


# ----------------------------------------------------------------------------
# Steps
# ----------------------------------------------------------------------------
def frame_positions(frame: int, tokens_per_frame: int, pos_offset: int = 0) -> np.ndarray:
    """Positions of frame ``frame``'s tokens from the virtual length L_n = pos_offset + frame*T
    (virtual sequence length paragraph): they do not depend on how many tokens C retains."""
    return pos_offset + frame * tokens_per_frame + np.arange(tokens_per_frame, dtype=np.int64)


def visibility(n_state: int, tokens_per_frame: int) -> np.ndarray:
    """Mask M_n of Eq. 5 as a [T, S+T] boolean array: memory tokens precede the frame and are
    visible to every frame query; inside the frame the mask is causal (key t visible iff t <= i)."""
    i = np.arange(tokens_per_frame)[:, None]
    j = np.arange(n_state + tokens_per_frame)[None, :]
    return (j < n_state) | ((j - n_state) <= i)


def kv_head_of(n_q_heads: int, n_kv_heads: int) -> np.ndarray:
    """Grouped-query attention: query head h reads KV head floor(h / G), G = H_q / H_kv."""
    return np.arange(n_q_heads) // (n_q_heads // n_kv_heads)


def frame_attention(q, k_pool, v_pool, n_state, scale):
    """Eq. 5: softmax(Q [K_state; K_frame]^T / sqrt(d_h) + M_n) [V_state; V_frame].

    q [H_q, T, d]; k_pool, v_pool [H_kv, S+T, d] (state first).  Returns (O, A) with
    A [H_q, T, S+T] the normalised attention (masked entries exactly 0)."""
    H_q, T, _ = q.shape
    H_kv = k_pool.shape[0]
    grp = kv_head_of(H_q, H_kv)
    K = k_pool[grp]
    V = v_pool[grp]
    logits = np.matmul(q, np.swapaxes(K, 1, 2)) * scale
    vis = visibility(n_state, T)
    logits = np.where(vis[None], logits, -np.inf)
    e = np.exp(logits - logits.max(axis=2, keepdims=True))
    A = e / e.sum(axis=2, keepdims=True)
    return np.matmul(A, V), A


def importance_scores(A, n_kv_heads):
    """s_{g,j} = (1/T) * sum_{h in group g} sum_i A_{h,i,j}  ->  [H_kv, S+T].

    The per-query average over the T frame queries is the paper's score
    instantiation; the group sum is the head aggregation done per KV head."""
    H_q, T, P = A.shape
    G = H_q // n_kv_heads
    return A.reshape(n_kv_heads, G, T, P).sum(axis=(1, 2)) / T


def select_top(scores, pos, capacity):
    """Eq. 6: indices of the ``capacity`` largest scores, ties broken by lowest position;
    everything is kept when the pool is not larger than the capacity.  Returned ascending
    in position."""
    P = scores.shape[0]
    if P <= capacity:
        keep = np.arange(P)
    else:
        order = np.lexsort((pos, -scores))  # primary key: score descending; secondary: position ascending
        keep = order[:capacity]
    return keep[np.argsort(pos[keep], kind="stable")]


def select_recent(pos, capacity):
    """Recency-window baseline: indices of the ``capacity`` largest positions (positions
    are distinct, so there are no ties); everything when the pool fits.  Ascending in
    position."""
    P = pos.shape[0]
    if P <= capacity:
        keep = np.arange(P)
    else:
        keep = np.argsort(-pos, kind="stable")[:capacity]
    return keep[np.argsort(pos[keep], kind="stable")]


POLICIES = ("statekv", "recent", "full")


def frame_step(state: LayerState, q, k, v, frame, capacity, scale=None, pos_offset=0,
               keep_attn=False, policy="statekv", rope: RopeSpec | None = None) -> StepResult:
    """One layer of one frame: attention over [C_{n-1}; frame], scores, refresh.

    q [H_q, T, d], k/v [H_kv, T, d] as float64 (exact widened input values).
    ``policy`` picks the refresh: "statekv" (Top-B by score, Eq. 6), "recent" (the B
    most recent candidates) or "full" (keep every candidate; ``capacity`` ignored, so
    the state is the whole token history and the step is streaming full attention).
    With ``rope``, Q and K are rotated at the frame's virtual positions first, and the
    rotated keys are what the state keeps (the state's keys are already rotated)."""
    if policy not in POLICIES:
        raise ValueError(f"unknown policy {policy!r}")
    H_q, T, d = q.shape
    H_kv = k.shape[0]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    S = state.size
    fpos = frame_positions(frame, T, pos_offset)
    if rope is not None:
        q = rope_rotate(q, fpos, rope)
        k = rope_rotate(k, fpos, rope)
    k_pool = np.concatenate([state.k, k], axis=1)
    v_pool = np.concatenate([state.v, v], axis=1)
    pool_pos = np.concatenate([state.pos, np.broadcast_to(fpos, (H_kv, T))], axis=1)

    out = np.empty_like(q)
    scores = np.empty((H_kv, S + T))
    attn = np.empty((H_q, T, S + T)) if keep_attn else None
    grp = kv_head_of(H_q, H_kv)
    for g in range(H_kv):  # one KV head at a time bounds memory; heads are independent
        hs = np.nonzero(grp == g)[0]
        o_g, a_g = frame_attention(q[hs], k_pool[g:g + 1], v_pool[g:g + 1], S, scale)
        out[hs] = o_g
        scores[g] = importance_scores(a_g, 1)[0]
        if keep_attn:
            attn[hs] = a_g

    if policy == "full":
        capacity = S + T
    n_keep = min(capacity, S + T)
    kept = np.empty((H_kv, n_keep), dtype=np.int64)
    for g in range(H_kv):
        if policy == "recent":
            kept[g] = select_recent(pool_pos[g], capacity)
        else:
            kept[g] = select_top(scores[g], pool_pos[g], capacity)
    rows = np.arange(H_kv)[:, None]
    new_state = LayerState(
        pos=pool_pos[rows, kept].copy(),
        k=k_pool[rows, kept].copy(),
        v=v_pool[rows, kept].copy(),
        score=scores[rows, kept].copy(),
    )
    flops = int(visibility(S, T).sum()) * H_q * 4 * d
    return StepResult(out, attn, pool_pos, scores, kept, new_state, flops, k)


@dataclass
class DecodeCache:
    """Detailed state D of one layer: every frame's K/V rows, in stream order (Eq. 4)."""

    k: list = field(default_factory=list)
    v: list = field(default_factory=list)

    def append(self, k, v):
        self.k.append(np.array(k, copy=True))
        self.v.append(np.array(v, copy=True))

    def as_arrays(self):
        return np.concatenate(self.k, axis=1), np.concatenate(self.v, axis=1)

    @property
    def n_tokens(self) -> int:
        return sum(x.shape[1] for x in self.k)


def run_layer(inputs, n_frames, capacity, n_kv_heads, head_dim, scale=None, pos_offset=0,
              state=None, start_frame=0, callback=None, policy="statekv", rope=None):
    """Stream ``n_frames`` frames of one layer.  ``inputs(frame)`` returns float64
    (q, k, v).  Returns (final state, decode cache, list of StepResult)."""
    st = state.copy() if state is not None else LayerState.empty(n_kv_heads, head_dim)
    cache = DecodeCache()
    results = []
    for n in range(start_frame, start_frame + n_frames):
        q, k, v = inputs(n)
        r = frame_step(st, q, k, v, n, capacity, scale, pos_offset, policy=policy, rope=rope)
        cache.append(r.k_stored, v)  # D_n = D_{n-1} with the frame's K/V appended
        st = r.state
        results.append(r if callback is None else callback(n, r))
    return st, cache, results


def decode_attention(q, k_hist, v_hist, k_new, v_new, scale=None, rope: RopeSpec | None = None, positions=None):
    """Decoding after (or between) frames reads the detailed state D, not C (the decoding
    paragraph): the t new tokens attend to every earlier token of D (the video's tokens, then
    the tokens decoded before), all visible, and to the new tokens up to themselves (causal).
    That is Eq. 5 with the whole history as the memory.

    q [H_q, t, d]; k_hist, v_hist [H_kv, n, d] (keys as D stores them); k_new, v_new
    [H_kv, t, d].  With ``rope``, the new tokens' Q and K are rotated at ``positions`` [t]
    first.  Returns [H_q, t, d]."""
    if rope is not None:
        q = rope_rotate(q, positions, rope)
        k_new = rope_rotate(k_new, positions, rope)
    H_q, t, d = q.shape
    H_kv = k_new.shape[0]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    n = k_hist.shape[1]
    k_pool = np.concatenate([k_hist, k_new], axis=1)
    v_pool = np.concatenate([v_hist, v_new], axis=1)
    out = np.empty_like(q)
    grp = kv_head_of(H_q, H_kv)
    for g in range(H_kv):
        hs = np.nonzero(grp == g)[0]
        out[hs] = frame_attention(q[hs], k_pool[g:g + 1], v_pool[g:g + 1], n, scale)[0]
    return out


def attention_flops(n_q_heads, head_dim, tokens_per_frame, n_state):
    """Closed form of StepResult.flops: 4*d*H_q*(T*S + T(T+1)/2)."""
    T = tokens_per_frame
    return 4 * head_dim * n_q_heads * (T * n_state + T * (T + 1) // 2)
