"""Brute-force checkers, written independently of the oracle.

* ``exact_topk`` ranks memory rows by their cosine score in exact rational
  arithmetic (Sec. 2.5, Tier-1 score): ||q|| is a positive constant, so the
  order of dot_j / ||m_j|| decides, and sign(dot)*dot^2/||m_j||^2 is an exact
  monotone stand-in for it.  Ties go to the lower index.
* ``history_attention`` keeps every sequence's token history as a Python
  list and takes "the last W tokens" by slicing: there is no ring
  arithmetic, so it checks the ring semantics as well as the attention
  (Sec. 2.5, KV cache assembly).  Logits and weights use Python floats with
  ``math.fsum``.

Pure-Python loops: small inputs only.
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import List, Sequence

import numpy as np


def exact_topk(keys: np.ndarray, q: np.ndarray, k: int) -> List[int]:
    """keys [N][D] fp32, q [D] fp32 -> the k best rows, ascending."""
    qf = [Fraction(float(x)) for x in np.asarray(q, np.float32)]
    q_zero = all(x == 0 for x in qf)
    ranked = []
    for j, row in enumerate(np.asarray(keys, np.float32)):
        mf = [Fraction(float(x)) for x in row]
        n2 = sum(a * a for a in mf)
        dot = sum(a * b for a, b in zip(mf, qf))
        if n2 == 0 or q_zero:
            key = Fraction(0)
        else:
            sign = (dot > 0) - (dot < 0)
            key = sign * dot * dot / n2
        ranked.append((key, j))
    ranked.sort(key=lambda t: (-t[0], t[1]))
    return sorted(j for _, j in ranked[:k])


def history_attention(q: np.ndarray, pool_k: np.ndarray, pool_v: np.ndarray,
                      rows: Sequence[int], hist_k: Sequence[list], hist_v: Sequence[list],
                      W: int, scale: float) -> np.ndarray:
    """One sequence.  q [Hq][Dh]; pool_* [Hkv][N][Dh] (float values);
    rows: the selected pool rows; hist_*[h]: list of token rows in arrival
    order for kv head h.  Returns [Hq][Dh] float64."""
    Hq, Dh = q.shape
    Hkv = pool_k.shape[0]
    G = Hq // Hkv
    out = np.zeros((Hq, Dh), np.float64)
    for h in range(Hq):
        kv = h // G
        window_k = list(hist_k[kv][-W:]) if W > 0 else []
        window_v = list(hist_v[kv][-W:]) if W > 0 else []
        keys = [pool_k[kv][r] for r in rows] + window_k
        vals = [pool_v[kv][r] for r in rows] + window_v
        if not keys:
            continue
        qh = [float(x) for x in q[h]]
        z = [scale * math.fsum(a * float(b) for a, b in zip(qh, key)) for key in keys]
        m = max(z)
        wts = [math.exp(t - m) for t in z]
        den = math.fsum(wts)
        for d in range(Dh):
            out[h, d] = math.fsum(wi * float(v[d]) for wi, v in zip(wts, vals)) / den
    return out
