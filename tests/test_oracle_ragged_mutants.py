"""The ragged pins reject plausible mistakes in the oracle's ragged
wrappers (planted in subclasses, on the CPU)."""
import numpy as np
import pytest

import oracle
from tests import pins


class _AllRows(oracle.Oracle):
    """Mistake: selects over all N rows instead of the first n_b."""

    def select_ragged(self, sel_keys, q_vec, n_rows, k, q_rows=None, idx_stride=None):
        return super().select_ragged(sel_keys, q_vec, np.full_like(n_rows, sel_keys.shape[1]), k, q_rows,
                                     idx_stride)


class _NoQuestion(oracle.Oracle):
    """Mistake: drops the pinned question rows."""

    def select_ragged(self, sel_keys, q_vec, n_rows, k, q_rows=None, idx_stride=None):
        return super().select_ragged(sel_keys, q_vec, n_rows, k, None, idx_stride)


class _UnclampedKlen(oracle.Oracle):
    """Mistake: a negative k_len is read as 'all k rows'."""

    def two_tier_decode_ragged(self, q, cme_k, cme_v, idx, k_len, k, *rest):
        return super().two_tier_decode_ragged(q, cme_k, cme_v, idx, np.where(k_len < 0, k, k_len), k, *rest)


class _UniformK(oracle.Oracle):
    """Mistake: every sequence uses all k pool rows."""

    def two_tier_decode_ragged(self, q, cme_k, cme_v, idx, k_len, k, *rest):
        return super().two_tier_decode_ragged(q, cme_k, cme_v, idx, np.full_like(k_len, k), k, *rest)


@pytest.mark.parametrize("cls,pin", [
    (_AllRows, pins.pin_select_ragged_brute),
    (_NoQuestion, pins.pin_select_ragged_brute),
    (_UnclampedKlen, pins.pin_decode_ragged_history),
    (_UniformK, pins.pin_decode_ragged_history),
])
def test_ragged_mutant_killed(cls, pin):
    bad = cls(oracle.build(force=False))
    with pytest.raises(AssertionError):
        pin(bad)
