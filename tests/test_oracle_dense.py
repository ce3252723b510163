"""Pins of the FC-DenseNet glue oracle (Section 6.2) against what fixes
each definition independently of its code: the L2 head gradient (already
pinned) for an infinite cutoff, finite differences of a separately written
Huber loss, exact saturation, brute-force pooling loops on tiny inputs,
the pooling adjoint identity on exactly representable values, and the
round trip of concatenation and slice reads."""
import numpy as np
import pytest

from oracle import dense as D
from oracle import grad as G


def _huber_mean(y, t, delta):
    # the loss written out per output: quadratic inside the cutoff, linear
    # beyond, averaged over the outputs
    d = y - t
    a = np.abs(d)
    return np.mean(np.where(a <= delta, 0.5 * d * d, delta * (a - 0.5 * delta)))


def test_infinite_cutoff_is_the_l2_gradient():
    rng = np.random.default_rng(1)
    y = rng.normal(size=(2, 8, 8, 1)).astype(np.float16)
    t = rng.normal(size=(2, 8, 8, 1)).astype(np.float32)
    S = 2.0 ** 15
    # mean((y-t)^2) has twice the gradient of mean(huber_inf)
    np.testing.assert_array_equal(D.huber_head_grad(y, t, 2 * S / y.size, np.inf),
                                  G.head_grad(y, t, S))


def test_huber_gradient_matches_finite_differences():
    rng = np.random.default_rng(2)
    n = 64
    t = rng.normal(size=n) * 20.0
    y = (t + rng.normal(size=n) * 15.0).astype(np.float16).astype(np.float64)
    delta = 10.0
    keep = np.abs(np.abs(y - t) - delta) > 1e-3   # away from the kink
    g = D.huber_head_grad(y.astype(np.float16), t.astype(np.float32), 1.0, delta)
    h = 1e-6
    tt = t.astype(np.float32).astype(np.float64)
    for j in np.nonzero(keep)[0][:32]:
        e = np.zeros(n)
        e[j] = h
        fd = (_huber_mean(y + e, tt, delta) - _huber_mean(y - e, tt, delta)) / (2 * h) * n
        assert float(g[j]) == pytest.approx(fd, rel=2e-3, abs=1e-6)


def test_huber_saturates_exactly():
    y = np.array([100.0, -100.0, 3.0, -10.0, 10.0], np.float16)
    t = np.zeros(5, np.float32)
    np.testing.assert_array_equal(D.huber_head_grad(y, t, 0.5, 10.0),
                                  np.array([5.0, -5.0, 1.5, -5.0, 5.0], np.float16))
    # scale large enough to overflow fp16 gives infinities of the right sign
    big = D.huber_head_grad(y, t, 1e5, 10.0)
    assert big[0] == np.inf and big[1] == -np.inf


def test_pooling_brute_force():
    rng = np.random.default_rng(3)
    x = rng.normal(size=(2, 4, 6, 3)).astype(np.float16)
    y = D.avg_pool2d_fwd(x)
    for n in range(2):
        for p in range(2):
            for q in range(3):
                for c in range(3):
                    s = sum(float(x[n, 2 * p + i, 2 * q + j, c]) for i in range(2) for j in range(2))
                    assert y[n, p, q, c] == np.float16(s / 4.0)
    dy = rng.normal(size=y.shape).astype(np.float16)
    gate = rng.normal(size=x.shape).astype(np.float16)
    dx = D.avg_pool2d_bwd(dy, gate)
    for n in range(2):
        for h in range(4):
            for w in range(6):
                for c in range(3):
                    want = float(dy[n, h // 2, w // 2, c]) / 4.0 if gate[n, h, w, c] > 0 else 0.0
                    assert dx[n, h, w, c] == np.float16(want)


def test_pooling_adjoint_on_exact_values():
    rng = np.random.default_rng(4)
    x = (rng.integers(-64, 64, size=(2, 8, 10, 5)) / 8.0).astype(np.float16)
    dy = (rng.integers(-64, 64, size=(2, 4, 5, 5)) / 8.0).astype(np.float16)
    lhs = np.sum(D.avg_pool2d_fwd(x).astype(np.float64) * dy.astype(np.float64))
    rhs = np.sum(x.astype(np.float64) * D.avg_pool2d_bwd(dy).astype(np.float64))
    assert lhs == rhs
    const = np.full((1, 6, 6, 4), 0.375, np.float16)
    assert np.all(D.avg_pool2d_fwd(const) == np.float16(0.375))


def test_concat_slices_round_trip_and_accumulate():
    rng = np.random.default_rng(5)
    pieces = [rng.normal(size=(2, 3, 3, c)).astype(np.float16) for c in (8, 16, 8)]
    z = D.concat_channels(pieces)
    assert z.shape == (2, 3, 3, 32)
    flat = z.reshape(-1, 32)
    off = 0
    for p in pieces:
        c = p.shape[-1]
        got = D.channel_slice_copy(flat[:, off:off + c], np.zeros((18, c), np.float16))
        np.testing.assert_array_equal(got, p.reshape(-1, c))
        off += c
    a = rng.normal(size=(18, 8)).astype(np.float16)
    b = rng.normal(size=(18, 8)).astype(np.float16)
    gate = rng.normal(size=(18, 8)).astype(np.float16)
    acc = D.channel_slice_copy(a, b, gate, accumulate=True)
    for i in range(18):
        for k in range(8):
            want = float(b[i, k]) + (float(a[i, k]) if gate[i, k] > 0 else 0.0)
            assert acc[i, k] == np.float16(want)
    big = np.full((1, 8), 60000, np.float16)
    assert np.all(D.channel_slice_copy(big, big, accumulate=True) == np.inf)
