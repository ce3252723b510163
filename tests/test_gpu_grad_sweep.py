"""Seeded random sweep of the gradient path (Section 4.2 grouping into a
fused buffer; Section 6.2 loss-scale unscaling with the overflow check)
against the NumPy oracle.

Each case draws a gradient set and a plan nobody picked: 1 to 64 members
(the most one call takes) of 1 to ~300k elements, a group capacity from
256 B to 4 MiB and an alignment of 16 B to 4 KiB, so that groups hold one
member or many, members larger than the capacity get groups of their own,
and the padding between members varies. Values are fp16 bit patterns of
every finite exponent, with seeded injections of +-inf, NaNs of several
payloads, subnormals, +-0 and +-65504; the inverse loss scale is a power of
two or an arbitrary fp32 value. Every buffer (sources, group, fp32 group,
destinations) is a view at a random element offset into a larger
allocation, so the vector and element-wise paths both run.

Bars: the packed group bit for bit (padding zero); unscaled and unpacked
fp32 values bit for bit where finite and class-exact where not (+-inf by
sign, NaN as NaN); the overflow flag exactly the oracle's.
"""
import zlib

import numpy as np
import pytest
import torch

import paper_1909_11150_amd as fg
from gpu_util import host
from oracle import grad as G

pytestmark = pytest.mark.gpu

SPECIALS = np.array([0x7C00, 0xFC00, 0x7E00, 0x7C01, 0xFFFF, 0x0001, 0x83FF,
                     0x0000, 0x8000, 0x7BFF, 0xFBFF], dtype=np.uint16)
NONFINITE = {0x7C00, 0xFC00, 0x7E00, 0x7C01, 0xFFFF}


def draw_case(i):
    rng = np.random.default_rng(zlib.crc32(f"grad-sweep-{i}".encode()))
    m = int(rng.integers(1, 65))
    numels = [int(v) for v in np.exp(rng.uniform(0, np.log(3e5), size=m)).astype(int) + 1]
    cap = int(np.exp(rng.uniform(np.log(256), np.log(4 << 20))))
    align = int(rng.choice((16, 64, 256, 4096)))
    inv = (np.float32(2.0 ** -int(rng.integers(0, 25))) if rng.random() < 0.5
           else np.float32(rng.uniform(1e-6, 1.0)))
    # about a third of the cases carry no non-finite value at all
    n_inject = 0 if i % 3 == 0 else int(rng.integers(1, 6))
    return rng, numels, cap, align, inv, n_inject


def _bits(rng, n):
    return (rng.integers(0, 0x7C00, size=n, dtype=np.uint16) |
            (rng.integers(0, 2, size=n, dtype=np.uint16) << 15))


def _view(n, dtype, rng, fill):
    """A length-n view at a random element offset 0..7 into a larger tensor
    filled with `fill`."""
    o = int(rng.integers(0, 8))
    return torch.full((n + 8,), fill, dtype=dtype, device="cuda")[o:o + n]


def _class_equal(got, ref, what):
    fin = np.isfinite(ref)
    np.testing.assert_array_equal(got[fin].view(np.uint32), ref[fin].view(np.uint32),
                                  err_msg=what)
    for pred in (np.isnan, np.isposinf, np.isneginf):
        np.testing.assert_array_equal(pred(got), pred(ref), err_msg=what)


@pytest.mark.parametrize("i", range(40))
def test_random_gradient_groups(i):
    rng, numels, cap, align, inv, n_inject = draw_case(i)
    print(f"case {i}: {len(numels)} members, {sum(numels)} elements, cap {cap} B, "
          f"align {align} B, inv {inv!r}, {n_inject} injections", flush=True)
    srcs = [_bits(rng, n) for n in numels]
    # special values at seeded (member, position) pairs, non-finite ones
    # only in the cases that inject
    for _ in range(n_inject + int(rng.integers(0, 6))):
        mbr = int(rng.integers(0, len(numels)))
        word = int(rng.choice(SPECIALS))
        if n_inject == 0 and word in NONFINITE:
            continue
        srcs[mbr][int(rng.integers(0, numels[mbr]))] = word
    plan = G.plan_groups(numels, cap, align)
    assert sum(len(g["members"]) for g in plan) == len(numels)
    dsrc = []
    for s in srcs:
        v = _view(s.size, torch.int16, rng, 0)
        v.copy_(torch.from_numpy(s.view(np.int16)))
        dsrc.append(v)
    for gi, grp in enumerate(plan):
        what = f"case {i} group {gi}"
        gbuf = _view(grp["numel"], torch.int16, rng, 0x5555)
        fg.grad_group_pack([dsrc[m] for m in grp["members"]], grp["offsets"], gbuf)
        g32 = _view(grp["numel"], torch.float32, rng, 7.0)
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        fg.grad_unscale_check(gbuf, inv, g32, flag)
        dsts = [_view(numels[m], torch.float32, rng, float("nan")) for m in grp["members"]]
        fg.grad_group_unpack(g32, dsts, grp["offsets"])
        ref16 = G.pack(srcs, grp)
        np.testing.assert_array_equal(host(gbuf).view(np.uint16), ref16, err_msg=what)
        r32, rflag = G.unscale_check(ref16, inv)
        assert int(host(flag)[0]) == int(rflag), what
        _class_equal(host(g32), r32, what)
        ref_out = G.unpack(r32, grp, numels)
        for m, d in zip(grp["members"], dsts):
            _class_equal(host(d), ref_out[m], f"{what} member {m}")
