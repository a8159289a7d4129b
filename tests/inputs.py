"""Test-side input preparation: the generator's draws plus the selection
gap rule, which needs the oracle's scores and therefore lives with the tests
rather than in the generator."""
from __future__ import annotations

from typing import List

import numpy as np

from paper_2609_25537_amd import workloads as wl


def accepted_attempts(w: wl.Workload, orc, max_attempts: int = 400) -> List[int]:
    """Per sequence, the first q_vec draw whose k-th/(k+1)-th score gap is at
    least w.gap_min (relative), so that the top-k set is decided the same
    way in fp32 and fp64."""
    out = []
    for b in range(w.B):
        keys = wl.sel_keys(w, b)[None]
        for a in range(max_attempts):
            _, _, gap = orc.select(keys, wl.q_vec(w, b, a)[None], w.k)
            if gap[0] >= w.gap_min:
                out.append(a)
                break
        else:
            raise RuntimeError(f"no draw with gap >= {w.gap_min} for sequence {b}")
    return out
