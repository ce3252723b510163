"""GPU parity of the gradient path (bit-exact) against the NumPy oracle."""
import numpy as np
import pytest
import torch

import paper_1909_11150_amd as fg
import synth
from gpu_util import dev, host
from oracle import grad as G

pytestmark = pytest.mark.gpu

INV = np.float32(2.0 ** -15)


def _rand16(rng, n):
    """fp16 bit patterns: finite values of every exponent, both signs."""
    return rng.integers(0, 0x7C00, size=n, dtype=np.uint16) | \
        (rng.integers(0, 2, size=n, dtype=np.uint16) << 15)


def _run_group(srcs16, grp, numels, inv=INV):
    """pack -> unscale_check -> unpack on the GPU for one planned group."""
    dsrc = [dev(s.view(np.int16)) for s in srcs16]
    members = [dsrc[m] for m in grp["members"]]
    gbuf = torch.full((grp["numel"],), 0x5555, dtype=torch.int16, device="cuda")
    fg.grad_group_pack(members, grp["offsets"], gbuf)
    g32 = torch.empty(grp["numel"], dtype=torch.float32, device="cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    fg.grad_unscale_check(gbuf, inv, g32, flag)
    dsts = [torch.full((numels[m],), float("nan"), dtype=torch.float32, device="cuda")
            for m in grp["members"]]
    fg.grad_group_unpack(g32, dsts, grp["offsets"])
    return (host(gbuf).view(np.uint16), host(g32), int(host(flag)[0]),
            {m: host(d) for m, d in zip(grp["members"], dsts)})


@pytest.mark.parametrize("numels,cap", [
    ([3, 700, 129, 64, 1000], 2048),
    ([8, 16, 24], 4096),
    ([1, 1, 1, 1], 256),
    ([100_003, 77, 250_000], 1 << 20),
])
def test_pack_unscale_unpack_bit_exact(numels, cap):
    rng = np.random.default_rng(sum(numels))
    srcs = [_rand16(rng, n) for n in numels]
    for grp in G.plan_groups(numels, cap, 256):
        buf, g32, flag, out = _run_group(srcs, grp, numels)
        ref = G.pack(srcs, grp)
        np.testing.assert_array_equal(buf, ref)
        r32, rflag = G.unscale_check(ref, INV)
        np.testing.assert_array_equal(g32.view(np.uint32), r32.view(np.uint32))
        assert flag == int(rflag) == 0
        for m, v in G.unpack(r32, grp, numels).items():
            np.testing.assert_array_equal(out[m].view(np.uint32), v.view(np.uint32))


@pytest.mark.parametrize("word,flag", [
    (None, 0), (0x7C00, 1), (0xFC00, 1), (0x7E00, 1), (0x7C01, 1),
    (0x7BFF, 0), (0x0001, 0), (0x8001, 0)])
@pytest.mark.parametrize("pos", ["first", "last", "tail", "middle"])
def test_fault_matrix(word, flag, pos):
    n = 4099  # not a multiple of the 8-element vector: exercises the tail
    buf = np.full(n, 0x3C00, np.uint16)
    i = {"first": 0, "last": n - 1, "tail": n - 2, "middle": 2048}[pos]
    if word is not None:
        buf[i] = word
    g = dev(buf.view(np.int16))
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    f = torch.zeros(1, dtype=torch.int32, device="cuda")
    fg.grad_unscale_check(g, INV, out, f)
    assert int(host(f)[0]) == flag
    ref, rflag = G.unscale_check(buf, INV)
    assert int(rflag) == flag
    got = host(out)
    fin = np.isfinite(ref)
    np.testing.assert_array_equal(got[fin].view(np.uint32), ref[fin].view(np.uint32))
    # non-finite outputs: class-exact (+-inf sign-exact, NaN any payload)
    np.testing.assert_array_equal(np.isnan(got), np.isnan(ref))
    np.testing.assert_array_equal(np.isposinf(got), np.isposinf(ref))
    np.testing.assert_array_equal(np.isneginf(got), np.isneginf(ref))


def test_flag_is_only_ever_set():
    """A clean buffer leaves a flag that is already 1 untouched."""
    g = dev(np.full(1000, 0x3C00, np.uint16).view(np.int16))
    out = torch.empty(1000, dtype=torch.float32, device="cuda")
    f = torch.ones(1, dtype=torch.int32, device="cuda")
    fg.grad_unscale_check(g, INV, out, f)
    assert int(host(f)[0]) == 1


@pytest.mark.parametrize("inv", [np.float32(1 / 3), np.float32(0.1)])
def test_unscale_any_scale_single_rounding(inv):
    rng = np.random.default_rng(3)
    b = _rand16(rng, 1 << 16)
    out = torch.empty(b.size, dtype=torch.float32, device="cuda")
    f = torch.zeros(1, dtype=torch.int32, device="cuda")
    fg.grad_unscale_check(dev(b.view(np.int16)), inv, out, f)
    np.testing.assert_array_equal(host(out).view(np.uint32),
                                  G.unscale(b, inv).view(np.uint32))


def test_misaligned_buffers():
    """Sub-views that are not 16-byte aligned take the element-wise path."""
    rng = np.random.default_rng(4)
    b = _rand16(rng, 1001)
    base = dev(np.concatenate([[0], b]).astype(np.uint16).view(np.int16))
    src = base[1:]
    gbuf = torch.zeros(1003, dtype=torch.int16, device="cuda")[1:1002]
    fg.grad_group_pack([src], [0], gbuf)
    np.testing.assert_array_equal(host(gbuf).view(np.uint16), b)
    o = torch.empty(1002, dtype=torch.float32, device="cuda")[1:]
    f = torch.zeros(1, dtype=torch.int32, device="cuda")
    fg.grad_unscale_check(gbuf, INV, o, f)
    np.testing.assert_array_equal(host(o).view(np.uint32), G.unscale(b, INV).view(np.uint32))
    d = torch.empty(1002, dtype=torch.float32, device="cuda")[1:]
    fg.grad_group_unpack(o, [d], [0])
    np.testing.assert_array_equal(host(d).view(np.uint32), G.unscale(b, INV).view(np.uint32))


def test_full_network_gradient_path_with_injection():
    """The 13 weight-gradient tensors of the full network (99,483,904 fp16
    values), 99 +inf injections at seeded positions before pack, the nine
    25 MiB groups: pack and unpack bit-exact, flags exact per group."""
    layers = synth.fcn_layers()
    order = list(reversed(range(len(layers))))
    numels = [layers[i].w_numel for i in order]
    rng = np.random.default_rng(12)
    srcs = [synth.normal(rng, (n,), 1.0).view(np.uint16) for n in numels]
    flat = np.concatenate(srcs)
    inj = synth.injection_indices(flat.size)
    flat[inj] = 0x7C00
    bounds = np.cumsum([0] + numels)
    srcs = [flat[bounds[i]:bounds[i + 1]] for i in range(len(numels))]
    plan = G.plan_groups(numels, synth.GROUP_CAP_BYTES, synth.GROUP_ALIGN_BYTES)
    gof, oof, gnum = fg.grad_group_plan(numels, synth.GROUP_CAP_BYTES, 256, 2)
    assert gnum == [p["numel"] for p in plan]
    assert len(plan) == 9
    for grp in plan:
        buf, g32, flag, out = _run_group(srcs, grp, numels)
        ref = G.pack(srcs, grp)
        assert np.array_equal(buf, ref)
        r32, rflag = G.unscale_check(ref, INV)
        assert flag == int(rflag)
        assert np.array_equal(g32.view(np.uint32), r32.view(np.uint32))
        for m, v in G.unpack(r32, grp, numels).items():
            assert np.array_equal(out[m].view(np.uint32), v.view(np.uint32))
    # every group holding an injected index is flagged; the rest are not
    hit = set(int(np.searchsorted(bounds, i, side="right") - 1) for i in inj)
    flagged = [any(m in hit for m in p["members"]) for p in plan]
    assert any(flagged)


def test_head_grad_bit_exact():
    rng = np.random.default_rng(5)
    y = synth.normal(rng, (4, 256, 256, 1), 2.0)
    t = synth.smooth_target(4, 256)
    dy = torch.empty(y.shape, dtype=torch.float16, device="cuda")
    scale = 2.0 * 2.0 ** 15 / y.size
    fg.l2_head_grad(dev(y), dev(t), scale, dy)
    ref = G.head_grad(y, t, 2.0 ** 15)
    np.testing.assert_array_equal(host(dy).view(np.uint16), ref.view(np.uint16))


def test_head_grad_rounding_edge_cases():
    # values chosen so that scale*(y - t) hits fp16 ties, subnormals, overflow
    y = np.array([1.0, 1.0, 0.0, 60000.0, -60000.0, 0.0, 2.0, 0.0], np.float16)
    t = np.array([1.0 - 2 ** -11, 1.0 - 3 * 2 ** -11, -(2 ** -25),
                  -60000.0, 60000.0, 2 ** -24 * 3, 2.0, 1e-30], np.float32)
    scale = 1.0
    dy = torch.empty(y.shape, dtype=torch.float16, device="cuda")
    fg.l2_head_grad(dev(y), dev(t), scale, dy)
    with np.errstate(over="ignore"):
        ref = ((y.astype(np.float64) - t.astype(np.float64)) * scale).astype(np.float16)
    np.testing.assert_array_equal(host(dy).view(np.uint16), ref.view(np.uint16))


def test_relu_backward_bit_exact():
    rng = np.random.default_rng(6)
    dy = synth.uniform(rng, (8, 64, 64, 128))
    a = synth.uniform(rng, dy.shape)
    out = torch.empty(dy.shape, dtype=torch.float16, device="cuda")
    fg.relu_backward(dev(dy), dev(a), out)
    np.testing.assert_array_equal(host(out).view(np.uint16),
                                  G.relu_backward(dy, a).view(np.uint16))


def test_empty_members():
    """Members with no elements (allowed, null or not): pack copies the
    others and zero-fills every uncovered element, the empty members
    included; unpack writes only the non-empty destinations; a group of
    empty members only packs to zeros and unpacks nothing."""
    rng = np.random.default_rng(12)
    numels = [0, 5, 0, 1000, 0]
    srcs = [_rand16(rng, n) for n in numels]
    offsets = [0, 8, 16, 24, 1030]
    grp = {"members": list(range(5)), "offsets": offsets, "numel": 1040}
    dsrc = [dev(s.view(np.int16)) if s.size else torch.empty(0, dtype=torch.int16,
                                                              device="cuda")
            for s in srcs]
    gbuf = torch.full((1040,), 0x5555, dtype=torch.int16, device="cuda")
    fg.grad_group_pack(dsrc, offsets, gbuf)
    ref = G.pack(srcs, grp)
    np.testing.assert_array_equal(host(gbuf).view(np.uint16), ref)
    g32 = torch.empty(1040, dtype=torch.float32, device="cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    fg.grad_unscale_check(gbuf, INV, g32, flag)
    dsts = [torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
            for n in numels]
    fg.grad_group_unpack(g32, dsts, offsets)
    r32, _ = G.unscale_check(ref, INV)
    for m, v in G.unpack(r32, grp, numels).items():
        np.testing.assert_array_equal(host(dsts[m]).view(np.uint32), v.view(np.uint32))
    # only empty members
    g2 = torch.full((64,), 0x5555, dtype=torch.int16, device="cuda")
    empty = [torch.empty(0, dtype=torch.int16, device="cuda")] * 2
    fg.grad_group_pack(empty, [0, 32], g2)
    assert not host(g2).any()
    e32 = [torch.empty(0, dtype=torch.float32, device="cuda")] * 2
    fg.grad_group_unpack(torch.zeros(64, dtype=torch.float32, device="cuda"), e32, [0, 32])
    torch.cuda.synchronize()
