"""Test-side input preparation: the generator's draws plus the selection
gap rule, which needs the oracle's scores and therefore lives with the tests
rather than in the generator."""
from __future__ import annotations

from typing import List

import numpy as np

from paper_2609_25537_amd import workloads as wl


def accepted_attempts(w: wl.Workload, orc, max_attempts: int = 400, batch: int = 32) -> List[int]:
    """Per sequence, the first q_vec draw whose k-th/(k+1)-th score gap is at
    least w.gap_min (relative), so that the top-k set is decided the same
    way in fp32 and fp64 (a ragged sequence: over its own n_b rows, k_b =
    min(k, n_b)).  Candidate draws are screened `batch` at a time
    with one fp64 matrix product; the accepted draw is confirmed with the
    oracle's own gap."""
    out = []
    n_rows = wl.ragged_sizes(w)["n_rows"]
    for b in range(w.B):
        nb = int(n_rows[b])
        kb = min(w.k, nb)  # a ragged sequence chooses among its own rows only
        keys = wl.sel_keys(w, b)[:nb]
        k64 = keys.astype(np.float64)
        inv_norm = 1.0 / np.maximum(np.sqrt((k64 * k64).sum(1)), 1e-8)
        found = None
        for a0 in range(0, max_attempts, batch):
            Q = np.stack([wl.q_vec(w, b, a) for a in range(a0, a0 + batch)]).astype(np.float64)
            S = (k64 @ Q.T) * inv_norm[:, None] / np.maximum(np.sqrt((Q * Q).sum(1)), 1e-8)[None, :]
            top = -np.partition(-S, (kb - 1, kb), axis=0)[[kb - 1, kb]] if 0 < kb < nb else None
            for j in range(batch):
                if top is None or (top[0, j] - top[1, j]) / abs(top[0, j]) >= 0.9 * w.gap_min:
                    _, _, gap = orc.select(keys[None], wl.q_vec(w, b, a0 + j)[None], kb)
                    if gap[0] >= w.gap_min:
                        found = a0 + j
                        break
            if found is not None:
                break
        if found is None:
            raise RuntimeError(f"no draw with gap >= {w.gap_min} for sequence {b}")
        out.append(found)
    return out
