"""The oracle against its pins (closed forms, brute force, library special
cases, invariants).  CPU only."""
import pytest

from tests import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_select_rejects_bad_k(orc):
    import numpy as np
    import oracle
    with pytest.raises(oracle.OracleError):
        orc.select(np.zeros((1, 4, 2), np.float32), np.ones((1, 2), np.float32), 5)


def test_decode_rejects_out_of_range_index(orc):
    import numpy as np
    import oracle
    q = np.ones((1, 1, 4), np.float32)
    pk = np.ones((1, 1, 3, 4), np.float32)
    with pytest.raises(oracle.OracleError):
        orc.two_tier_decode(q, pk, pk, np.array([[3]], np.int32), 1, None, None, None, 0, 1.0)
