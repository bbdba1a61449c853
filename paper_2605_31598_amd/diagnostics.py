"""Assumption diagnostics of the method (appendix: concentration of inter-frame
attention, slow evolution of the temporal state), computed from the layer-level
attention scores the library reports.

For frame n of one layer, s_{n,j} is the attention mass key j receives from the
frame's queries, summed over every query head (the appendix's layer-level
score).  Run with a capacity at least as large as the stream (every earlier
token stays a candidate), the library's per-KV-head importance scores of frame
n cover exactly the keys a full-history frame attends to, and their sum over
KV heads, times T, is s_{n,j}.

* Concentration: the share of the historical attention mass (keys of frames
  < n) held by the B historical keys with the largest s_{n,j}.
* Candidate-pool recall: with S_n the top-B keys of all tokens seen up to frame
  n ranked by s_{n,j} (the oracle state), the share of S_{n+1} found in
  S_n u frame_{n+1}; weighted by s_{n+1,j}.
* Retention |S_n n S_{n+1}| / |S_n| and churn |S_{n+1} \\ S_n| / |S_{n+1}|.

Ties in a top-B are broken by the lower position, as in the selection rule.
"""
from __future__ import annotations

import numpy as np


def top_b(scores, positions, budget):
    """Positions of the `budget` largest scores (ties: lower position)."""
    if budget >= scores.shape[0]:
        return set(int(p) for p in positions)
    order = np.lexsort((positions, -scores))
    return set(int(p) for p in positions[order[:budget]])


def concentration(scores, positions, first_frame_pos, budget):
    """Share of the historical mass (keys before the frame) in its top-`budget` keys."""
    hist = positions < first_frame_pos
    s, p = scores[hist], positions[hist]
    total = s.sum()
    if total <= 0 or s.size == 0:
        return float("nan")
    keep = top_b(s, p, budget)
    mask = np.isin(p, np.fromiter(keep, dtype=np.int64, count=len(keep)))
    return float(s[mask].sum() / total)


def evolution(prev_scores, prev_pos, scores, pos, frame_pos, budget):
    """Recall, weighted recall, retention and churn between consecutive oracle states.

    prev_*: layer scores of frame n over all tokens seen up to frame n; scores/pos: of
    frame n+1 over all tokens up to frame n+1; frame_pos: positions of frame n+1."""
    s_prev = top_b(prev_scores, prev_pos, budget)
    s_next = top_b(scores, pos, budget)
    pool = s_prev | set(int(p) for p in frame_pos)
    hit = s_next & pool
    w = dict(zip((int(p) for p in pos), scores))
    w_all = sum(w[p] for p in s_next)
    return {
        "recall": len(hit) / len(s_next),
        "weighted_recall": (sum(w[p] for p in hit) / w_all) if w_all > 0 else float("nan"),
        "retention": len(s_prev & s_next) / len(s_prev),
        "churn": len(s_next - s_prev) / len(s_next),
    }


def summarise(frames, budgets):
    """frames: list over n of (scores [K], positions [K], first position of frame n), the layer
    scores of frame n over every token seen up to and including frame n.  Returns the means over
    frames of every diagnostic, per budget."""
    out = {}
    for b in budgets:
        conc = [concentration(s, p, f0, b) for s, p, f0 in frames[1:]]
        evo = [evolution(frames[n][0], frames[n][1], frames[n + 1][0], frames[n + 1][1],
                         frames[n + 1][1][frames[n + 1][1] >= frames[n + 1][2]], b)
               for n in range(len(frames) - 1)]
        out[b] = {"concentration": float(np.nanmean(conc)),
                  **{k: float(np.nanmean([e[k] for e in evo])) for k in evo[0]}}
    return out


def layer_frames_from_stepper(stepper, layer, tokens_per_frame):
    """Layer scores (summed over KV heads, times T) and positions of the last step's pool,
    read from a stepper whose capacity keeps every token (the pool is the whole history)."""
    st = stepper.read_state(layer)
    pos = st["pool_pos"][0].astype(np.int64)
    if not all(np.array_equal(st["pool_pos"][g], st["pool_pos"][0]) for g in range(st["pool_pos"].shape[0])):
        raise ValueError("pools differ between KV heads: the capacity does not keep every token")
    s = st["pool_score"].astype(np.float64).sum(axis=0) * tokens_per_frame
    return s, pos
