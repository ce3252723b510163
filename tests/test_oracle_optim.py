"""Pins of the optimizer oracle (layer-wise adaptive Adam, loss-scale
backoff; Section 6.2) against properties that fix each part of its
definition: closed forms of the first step, the norm of every layer's step,
Adam's invariance to the gradient's scale, exact bias correction under a
constant gradient, weight decay alone, the zero-weight fallback, and a
hand-traced loss-scale sequence."""
import math

import numpy as np
import pytest

from oracle import optim as O


def test_first_step_closed_form():
    # t = 1 from zero moments: m^ = g, v^ = g^2, so u = sign(g) with eps = 0;
    # ||w|| = 5 and ||u|| = sqrt(3) give tau = 5 / sqrt(3)
    w = np.array([3.0, 4.0, 0.0])
    g = np.array([1.0, -2.0, 0.5])
    lr = 0.01
    w1, m1, v1, tau = O.lars_adam_update(w, np.zeros(3), np.zeros(3), g, 1, lr,
                                         eps=0.0, wd=0.0)
    s = lr * 5.0 / math.sqrt(3.0)
    np.testing.assert_allclose(w1, [3.0 - s, 4.0 + s, -s], rtol=0, atol=1e-15)
    np.testing.assert_allclose(m1, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v1, 0.001 * g * g, rtol=1e-12)
    assert tau == pytest.approx(5.0 / math.sqrt(3.0), rel=1e-15)


def test_every_layer_step_has_norm_lr_times_weight_norm():
    rng = np.random.default_rng(3)
    for _ in range(5):
        n = int(rng.integers(2, 200))
        w, g = rng.normal(size=n), rng.normal(size=n) * 10.0 ** rng.integers(-6, 3)
        m, v = rng.normal(size=n) * 1e-3, rng.random(n) * 1e-4
        lr = 10.0 ** rng.uniform(-5, -1)
        w1, _, _, _ = O.lars_adam_update(w, m, v, g, int(rng.integers(1, 50)), lr)
        assert np.linalg.norm(w - w1) == pytest.approx(lr * np.linalg.norm(w), rel=1e-12)


def test_update_does_not_depend_on_gradient_scale():
    # Adam normalizes by the second moment: scaling g by c > 0 (no weight
    # decay, eps = 0, fresh moments) changes neither the step nor tau
    rng = np.random.default_rng(4)
    w, g = rng.normal(size=64), rng.normal(size=64)
    a = O.lars_adam_update(w, np.zeros(64), np.zeros(64), g, 1, 1e-3, eps=0.0, wd=0.0)
    b = O.lars_adam_update(w, np.zeros(64), np.zeros(64), 1e-4 * g, 1, 1e-3, eps=0.0, wd=0.0)
    np.testing.assert_allclose(a[0], b[0], rtol=1e-13)


def test_constant_gradient_gives_sign_steps_at_every_t():
    # bias correction makes m^ = g and v^ = g^2 exactly for a constant g, so
    # each step is lr * ||w_t|| * sign(g) / sqrt(n)
    w = np.array([1.0, -2.0, 0.5, 4.0])
    g = np.array([0.3, -0.1, 2.0, -5.0])
    m, v = np.zeros(4), np.zeros(4)
    lr = 0.05
    for t in range(1, 8):
        expect = w - lr * np.linalg.norm(w) * np.sign(g) / 2.0
        w, m, v, _ = O.lars_adam_update(w, m, v, g, t, lr, eps=0.0, wd=0.0)
        np.testing.assert_allclose(w, expect, rtol=1e-12, atol=1e-14)


def test_weight_decay_alone_shrinks_along_the_weights():
    # g = 0: the decayed gradient is wd * w, so u = sign(w) at t = 1
    w = np.array([2.0, -1.0, 0.25])
    w1, _, _, _ = O.lars_adam_update(w, np.zeros(3), np.zeros(3), np.zeros(3), 1, 0.1,
                                     eps=0.0, wd=1e-4)
    np.testing.assert_allclose(w1, w - 0.1 * np.linalg.norm(w) * np.sign(w) / math.sqrt(3),
                               rtol=1e-14)


def test_zero_weights_fall_back_to_a_unit_trust_ratio():
    w = np.zeros(2)
    g = np.array([1.0, -1.0])
    w1, _, _, tau = O.lars_adam_update(w, np.zeros(2), np.zeros(2), g, 1, 0.5, eps=0.0)
    assert tau == 1.0
    np.testing.assert_allclose(w1, [-0.5, 0.5], rtol=1e-15)


def test_fp16_copy_rounds_to_nearest_even():
    vals = np.array([1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, 65519.0, 65520.0])
    got = O.fp16_copy(vals)
    assert got[0] == 1.0 and got[1] == np.float16(1.0 + 2.0 ** -9)
    assert got[2] == 65504.0 and np.isposinf(got[3])


def test_loss_scale_backoff_sequence():
    # interval 3: overflow halves and skips; three clean steps double
    s, clean = 2.0 ** 15, 0
    seq = [False, True, False, False, False, False, True, True]
    trace = []
    for found in seq:
        s, clean, applied = O.loss_scale_next(s, clean, found, interval=3, s_min=2.0 ** 13)
        trace.append((s, clean, applied))
    assert trace == [(2.0 ** 15, 1, True), (2.0 ** 14, 0, False), (2.0 ** 14, 1, True),
                     (2.0 ** 14, 2, True), (2.0 ** 15, 0, True), (2.0 ** 15, 1, True),
                     (2.0 ** 14, 0, False), (2.0 ** 13, 0, False)]
    s, clean, _ = O.loss_scale_next(2.0 ** 13, 0, True, s_min=2.0 ** 13)
    assert s == 2.0 ** 13


def test_lr_schedule_hand_values():
    # warm-up 1e-4 -> 8e-4 over 7 updates: +1e-4 per update, exactly the
    # peak at k = 7; then x0.5 every 3 updates
    f = lambda k: O.lr_at(k, base=1e-4, peak=8e-4, warmup=7, every=3, rate=0.5)
    np.testing.assert_allclose([f(k) for k in range(7)],
                               [1e-4 * (1 + k) for k in range(7)], rtol=1e-14)
    assert [f(k) for k in (7, 8, 9, 10, 12, 13, 16)] == \
        [8e-4, 8e-4, 8e-4, 4e-4, 4e-4, 2e-4, 1e-4]
    # one rank, no warm-up, no decay: the paper's initial rate throughout
    assert {O.lr_at(k) for k in range(50)} == {1e-4}


def test_lr_schedule_shape():
    rng = np.random.default_rng(9)
    for _ in range(20):
        base = 10.0 ** rng.uniform(-5, -3)
        n = int(rng.integers(1, 64))
        wu, ev = int(rng.integers(1, 40)), int(rng.integers(1, 30))
        rate = float(rng.uniform(0.1, 0.99))
        lr = [O.lr_at(k, base, n * base, wu, ev, rate) for k in range(wu + 5 * ev)]
        d = np.diff(lr[:wu + 1])
        assert np.all(d >= 0) and np.allclose(d, d[0], rtol=1e-9)   # linear
        assert lr[wu] == n * base
        tail = np.array(lr[wu:])
        assert np.all(np.diff(tail) <= 0)                          # decays
        assert len(set(np.round(tail / (n * base), 12))) == 5      # 5 stairs
