"""The oracle against its pins (hand-worked fixtures, exhaustive scoring, closed forms,
invariants).  CPU only."""
import pytest

import oracle.umem_oracle as O
from tests.pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda p: getattr(p, "__name__", "pin"))
def test_pin(pin):
    pin(O)


def test_rejects_nan_and_degenerate_core():
    import numpy as np
    with pytest.raises(ValueError):
        O.top_sorted(np.array([1.0, np.nan]), 1)
    with pytest.raises(ValueError):
        O.rank1_factors(np.eye(2))        # sigma_1 == sigma_2: leading pair not unique
    with pytest.raises(ValueError):
        O.score_topk(np.zeros((1, 1, 2)), np.zeros((1, 1, 2)), np.zeros((1, 3, 2)),
                     np.zeros((1, 3, 2)), topk=2, topm=5)
