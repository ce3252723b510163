"""Pins for the grouping / pack / unscale / unpack oracle (CPU only)."""
import json
import os

import numpy as np
import pytest

import synth
from oracle import grad as G

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold_groups():
    with open(os.path.join(GOLD, "fcn_groups.json")) as f:
        return json.load(f)


def test_fcn_layer_table_matches_fixture():
    g = _gold_groups()
    layers = synth.fcn_layers()
    order = [L.name for L in reversed(layers)]
    assert order == g["completion_order"]
    assert [L.w_numel for L in reversed(layers)] == g["numels"]
    assert sum(g["numels"]) == 99_483_904


@pytest.mark.parametrize("cap", [25 * 1024 * 1024, 25_000_000])
def test_planner_gives_the_nine_groups(cap):
    g = _gold_groups()
    plan = G.plan_groups(g["numels"], cap, g["align_bytes"])
    names = g["completion_order"]
    got = [{"members": [names[m] for m in p["members"]], "numel": p["numel"]}
           for p in plan]
    assert got == g["groups"]


def test_planner_rules_on_small_cases():
    # alignment: 3 elements then 5 -> second member starts at 128 (256 B)
    p = G.plan_groups([3, 5], cap_bytes=1024, align_bytes=256)
    assert p == [{"members": [0, 1], "offsets": [0, 128], "numel": 133}]
    # close before overflow: 400 + aligned 128.. would pass 1024 B cap
    p = G.plan_groups([300, 300], cap_bytes=1024, align_bytes=256)
    assert [q["members"] for q in p] == [[0], [1]]
    # oversize singleton, then a fresh group
    p = G.plan_groups([10, 1000, 10], cap_bytes=256, align_bytes=256)
    assert [q["members"] for q in p] == [[0], [1], [2]]
    assert [q["numel"] for q in p] == [10, 1000, 10]
    # exactly at the cap still fits
    p = G.plan_groups([64, 64], cap_bytes=256 + 128, align_bytes=256)
    assert [q["members"] for q in p] == [[0, 1]]


def _rand16(rng, n):
    return rng.integers(0, 0x7C00, size=n, dtype=np.uint16) | \
        (rng.integers(0, 2, size=n, dtype=np.uint16) << 15)


def test_pack_unscale_unpack_round_trip():
    """unpack(unscale(pack(g))) = value(g) * 2^-15 exactly, per tensor, and
    the padding between members is zero."""
    rng = np.random.default_rng(5)
    numels = [3, 700, 129, 64, 1000]
    srcs = [_rand16(rng, n) for n in numels]
    plan = G.plan_groups(numels, cap_bytes=2048, align_bytes=256)
    inv = np.float32(2.0 ** -15)
    got = {}
    for grp in plan:
        buf = G.pack(srcs, grp)
        covered = np.zeros(grp["numel"], bool)
        for m, off in zip(grp["members"], grp["offsets"]):
            covered[off:off + numels[m]] = True
        assert np.all(buf[~covered] == 0)
        out, found = G.unscale_check(buf, inv)
        assert not found
        got.update(G.unpack(out, grp, numels))
    for i, s in enumerate(srcs):
        ref = np.ldexp(s.view(np.float16).astype(np.float32), -15)
        np.testing.assert_array_equal(got[i].view(np.uint32), ref.view(np.uint32))


def test_unscale_is_one_fp32_rounding_for_any_scale():
    """For inv_scale that is not a power of two, the fp64 route equals a
    single IEEE fp32 multiply (NumPy float32 arithmetic)."""
    rng = np.random.default_rng(6)
    b = _rand16(rng, 100_000)
    for inv in [np.float32(1 / 3), np.float32(0.1), np.float32(3.0e-5)]:
        ref = b.view(np.float16).astype(np.float32) * inv
        np.testing.assert_array_equal(G.unscale(b, inv).view(np.uint32),
                                      ref.view(np.uint32))


@pytest.mark.parametrize("word,flag", [
    (None, 0), (0x7C00, 1), (0xFC00, 1), (0x7E00, 1), (0x7C01, 1),
    (0x7BFF, 0), (0x0001, 0), (0x8001, 0), (0xFBFF, 0)])
@pytest.mark.parametrize("pos", ["first", "last", "tail"])
def test_fault_matrix(word, flag, pos):
    n = 1027
    buf = np.full(n, 0x3C00, np.uint16)
    if word is not None:
        i = {"first": 0, "last": n - 1, "tail": n - 3}[pos]
        buf[i] = word
    out, found = G.unscale_check(buf, np.float32(2.0 ** -15))
    assert found == bool(flag)
    if word in (0x0001, 0x8001):
        v = np.float16(0).view(np.uint16)
        i = {"first": 0, "last": n - 1, "tail": n - 3}[pos]
        expect = np.float32(np.ldexp(np.float64(2.0 ** -24), -15))
        assert out[i] == (expect if word == 0x0001 else -expect)
    if word == 0xFC00:
        i = {"first": 0, "last": n - 1, "tail": n - 3}[pos]
        assert np.isneginf(out[i])


def test_negative_zero_survives_unscale():
    out = G.unscale(np.array([0x8000, 0x0000], np.uint16), np.float32(2 ** -15))
    assert np.signbit(out[0]) and not np.signbit(out[1])


def test_injection_recipe():
    idx = synth.injection_indices(99_483_904)
    assert idx.size == 99 and np.unique(idx).size == 99
    assert idx.min() >= 0 and idx.max() < 99_483_904


def test_head_grad_rounding():
    """fp64 -> fp16 is one nearest-even rounding (no fp32 detour): a value
    just above a tie rounds up; the FCN factor 2*2^15/(4*256*256) = 1/4."""
    y = np.array([1.0 + 2 ** -11 + 2 ** -40], np.float64)
    assert y.astype(np.float16)[0] == np.float16(1.0 + 2 ** -10)
    assert np.float32(y[0]).astype(np.float16) == np.float16(1.0)
    y16 = np.array([[1.5, -2.0], [0.25, 8.0]], np.float16)
    t = np.array([[0.5, 2.0], [0.25, -8.0]], np.float32)
    dy = G.head_grad(y16, t, loss_scale=2.0)  # factor 2*2/4 = 1
    np.testing.assert_array_equal(dy, np.array([[1.0, -4.0], [0.0, 16.0]], np.float16))
    # overflow to infinity, no saturation
    assert np.isinf(G.head_grad(np.array([60000.0], np.float16),
                                np.array([-60000.0], np.float32), 1.0)[0])


def test_relu_backward():
    dy = np.array([1.0, -2.0, 3.0, -0.0], np.float16)
    a = np.array([0.5, 0.0, -1.0, 2.0], np.float16)
    r = G.relu_backward(dy, a)
    np.testing.assert_array_equal(r, np.array([1.0, 0.0, 0.0, -0.0], np.float16))
    assert not np.signbit(r[1]) and np.signbit(r[3])
