"""Brute-force StateKV frame step in pure Python loops, for tiny inputs.

TEST INFRASTRUCTURE ONLY (same import rule as the vectorised oracle).  Written
independently of ``statekv_oracle``: scalar loops, ``math.exp``, Python
``sorted``; it exists to pin the vectorised oracle on inputs small enough for
loops (a handful of heads, T <= 8, a few dozen candidates).

Definitions followed (Method, per-frame cache-builder forward pass):
* Eq. 5 with mask M_n: state keys always visible, frame key t visible to frame
  query i iff t <= i; logits scaled by ``scale``; query head h reads KV head h // G.
* Score of candidate j for KV head g: (1/T) times the attention mass it receives
  from all queries of the G query heads of group g.
* Eq. 6: keep the B highest scores, lower position first on equal scores.
"""
from __future__ import annotations

import math


def step(q, state, k, v, frame, capacity, scale, pos_offset=0):
    """q[h][i][e], k/v[g][t][e] nested lists of floats; state = list over KV heads of
    lists of (pos, krow, vrow).  Returns dict(out, scores, pool_pos, new_state)."""
    H_q = len(q)
    T = len(q[0])
    H_kv = len(k)
    G = H_q // H_kv
    out = [[None] * T for _ in range(H_q)]
    scores, pool_pos, new_state = [], [], []
    for g in range(H_kv):
        pool = list(state[g]) + [
            (pos_offset + frame * T + t, k[g][t], v[g][t]) for t in range(T)
        ]
        S = len(state[g])
        mass = [0.0] * len(pool)
        for h in range(g * G, (g + 1) * G):
            for i in range(T):
                vis = [j for j in range(len(pool)) if j < S or (j - S) <= i]
                logit = {}
                for j in vis:
                    dot = 0.0
                    for e in range(len(q[h][i])):
                        dot += q[h][i][e] * pool[j][1][e]
                    logit[j] = dot * scale
                top = max(logit.values())
                w = {j: math.exp(logit[j] - top) for j in vis}
                z = sum(w.values())
                row = [0.0] * len(pool[0][2])
                for j in vis:
                    a = w[j] / z
                    mass[j] += a
                    for e in range(len(row)):
                        row[e] += a * pool[j][2][e]
                out[h][i] = row
        s = [m / T for m in mass]
        ranked = sorted(range(len(pool)), key=lambda j: (-s[j], pool[j][0]))
        keep = ranked[: min(capacity, len(pool))]
        keep.sort(key=lambda j: pool[j][0])
        scores.append(s)
        pool_pos.append([p[0] for p in pool])
        new_state.append([(pool[j][0], pool[j][1], pool[j][2]) for j in keep])
    return {"out": out, "scores": scores, "pool_pos": pool_pos, "new_state": new_state}
