"""Seeded inputs with a peaked softmax over a long context ("attention sink").

One token of every kv-head's stream (the sink) receives a score ``gap`` log2
units above the bulk of the other scores for each query head of its group; the
other tokens' scores are tightly clustered around 0 (queries scaled by 1/4),
so that nearly all of them sit about ``gap`` binades below the sink. The value
channels of the other tokens have a nonzero mean (+-mu per channel) and the
sink's value vector is small, so that the output depends, at the 1e-3 level, on
the probability mass of the many small weights: a kernel that flushes small
probabilities to zero, or normalises by a sum other than the one it weights
the values with, misses it.

Data only: the sink key is a multiple of the sum of its group's queries, scaled
so that the smallest sink score of the group's heads is ``gap`` log2 units
(the bulk scores have median about 0); the test measures the gap it gets.
"""
from __future__ import annotations

import numpy as np

from paper_2505_22913_amd import synth

Q_SCALE = 0.25


def sink_case(B: int, Hkv: int, G: int, N: int, d: int, *, gap: float, late: bool, seed: int,
              mu: float = 3.0, sink_v_scale: float = 0.25, sK: float = 0.7):
    """(q [B][Hkv*G][d], K, V [B][Hkv][N][d] fp16, sink index). The query heads of
    a group share most of their direction, so their sink gaps are close."""
    K, V = synth.make_kv(B, Hkv, N, d, seed=seed)
    rng = np.random.default_rng(seed + 12345)
    own = synth.make_q(B, Hkv * G, d, seed=seed).astype(np.float32).reshape(B, Hkv, G, d)
    shared = rng.standard_normal((B, Hkv, 1, d)).astype(np.float32)
    q = ((shared + 0.25 * own) / np.sqrt(1.0625) * Q_SCALE).reshape(B, Hkv * G, d).astype(np.float16)
    sink = N - 100 if late else 5
    n_keep = d - int(np.floor(sK * d + 0.5))
    log2e = 1.4426950408889634
    Vf = V.astype(np.float32)
    for b in range(B):
        for h in range(Hkv):
            qg = q[b, h * G:(h + 1) * G].astype(np.float64)       # [G][d]
            u = qg.sum(axis=0)
            top = np.argsort(-np.abs(u), kind="stable")[:n_keep]   # channels the sink keeps
            per_head = (qg[:, top] @ u[top]) / np.sqrt(d) * log2e  # score per unit of alpha
            alpha = gap / per_head.min()
            K[b, h, sink] = (alpha * u).astype(np.float16)
            mean = mu * rng.choice([-1.0, 1.0], size=d)
            Vf[b, h] += mean
            Vf[b, h, sink] = sink_v_scale * rng.standard_normal(d)
    return q, K, Vf.astype(np.float16), sink
