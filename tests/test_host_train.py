"""Host logic of the training step (no GPU): the loss scaler and the
learning-rate schedule that the step program applies between steps follow
the oracle's backoff rule and schedule on random sequences, and reject
invalid parameters."""
import numpy as np
import pytest

from oracle import optim as O
from paper_1909_11150_amd.fcn import AdamLARS, LossScaler, LRSchedule


@pytest.mark.parametrize("interval", [1, 3, 2000])
def test_loss_scaler_follows_the_oracle(interval):
    rng = np.random.default_rng(interval)
    sc = LossScaler(2.0 ** 15, interval, s_min=2.0 ** 3, s_max=2.0 ** 17)
    s, c = 2.0 ** 15, 0
    for _ in range(3000):
        found = bool(rng.random() < 0.05)
        applied = sc.update(found)
        s, c, ok = O.loss_scale_next(s, c, found, interval, 2.0 ** 3, 2.0 ** 17)
        assert (sc.scale, sc.clean, applied) == (s, c, ok)


def test_loss_scaler_bounds_and_validation():
    sc = LossScaler(4.0, interval=1, s_min=2.0, s_max=8.0)
    assert [sc.update(True) or sc.scale for _ in range(3)] == [2.0, 2.0, 2.0]
    assert [sc.update(False) and sc.scale for _ in range(4)] == [4.0, 8.0, 8.0, 8.0]
    for bad in [dict(interval=0), dict(s_min=0.0), dict(scale=1.0, s_min=2.0),
                dict(scale=2.0 ** 30)]:
        with pytest.raises(ValueError):
            LossScaler(**bad)


def test_lr_schedule_follows_the_oracle():
    rng = np.random.default_rng(5)
    for _ in range(30):
        base = 10.0 ** rng.uniform(-5, -3)
        kw = dict(peak=base * int(rng.integers(1, 9)), warmup=int(rng.integers(0, 20)),
                  every=int(rng.integers(0, 10)), rate=float(rng.uniform(0.2, 1.0)))
        sch = LRSchedule(base, **kw)
        for k in range(100):
            assert sch(k) == pytest.approx(O.lr_at(k, base, **kw), rel=1e-12)
    with pytest.raises(ValueError):
        LRSchedule(warmup=-1)
    o = AdamLARS(lr=LRSchedule(1e-4, 4e-4, warmup=3))
    assert [o.lr_at(k) for k in range(4)] == pytest.approx([1e-4, 2e-4, 3e-4, 4e-4])
    assert AdamLARS(lr=3e-3).lr_at(10) == 3e-3
