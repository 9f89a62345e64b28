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


@pytest.mark.parametrize("pin", __import__("tests.pins", fromlist=["SCALE_PINS"]).SCALE_PINS,
                         ids=lambda p: p.__name__)
def test_pin_paper_scale(pin):
    pin(O)


@pytest.mark.parametrize("name", ["tucker-ive-4M", "tucker-ive-mcs-4M", "ultramem-1.6B-x12"])
def test_report_tucker_recall(name, capsys):
    """The recall of the rank-1 Tucker retrieval against the exhaustive exact-Tucker top-m on
    sampled tokens of the Tucker layers (reported, not asserted beyond its range)."""
    import dataclasses

    import numpy as np

    from synth import configs as CF
    from tests.pins import tucker_recall
    cfg = (dataclasses.replace(CF.C5, cores=2, name=name) if name == "tucker-ive-mcs-4M"
           else {c.name: c for c in (CF.C5, CF.C6)}[name])
    tokens = np.sort(np.random.default_rng(7).choice(cfg.T, 24, replace=False))
    rec = tucker_recall(O, cfg, tokens)
    assert ((rec >= 0) & (rec <= 1)).all()
    with capsys.disabled():
        print(f"\n[recall] {name}: rank-1 retrieval recall@{cfg.topm} of the exact Tucker top-"
              f"{cfg.topm} over {rec.size} (token, head) pairs: mean {rec.mean():.4f}, "
              f"min {rec.min():.4f}, max {rec.max():.4f}")
