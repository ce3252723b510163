"""Zero-copy gradient groups: conv2d_bwd_weight_checked.

The kernel gradient can write its fp16 dW straight into the member's slot of
its group buffer (the fusion buffer of Section 4.2 without the copy-in), and
flags a non-finite result in the same store (the check of Section 6.2's loss
scaling). Checks:
- the checked call writes bit for bit what conv2d_bwd_weight writes, on each
  kernel path (LDS-DMA with and without a split reduction, the register-
  staged kernel, the K = 1 head);
- a closed form pins both the values and the flag: with x = dy = a constant
  a, a 3x3 stride-1 pad-1 kernel gradient is a^2 * n * cnt(r) * cnt(s) with
  cnt = (h-1, h, h-1) by (w-1, w, w-1); a is a power of two chosen so that
  only the centre tap reaches 65520 (rounds to +inf in fp16) while every
  other tap stays finite, so the flag must be raised; at a / 2 nothing
  overflows and the flag must stay 0;
- a step with zero-copy groups gives the same master gradients and flags as
  a step that packs.
"""
import numpy as np
import pytest
import torch

import paper_1909_11150_amd as fg
import synth
from gpu_util import dev, empty16, host, workspace
from paper_1909_11150_amd.fcn import Chain

pytestmark = pytest.mark.gpu

# (n, h, w, c, k), kernel path
PATHS = [
    ((1, 16, 16, 256, 256), "wgrad_dma_kernel<false>"),
    ((4, 64, 64, 256, 256), "wgrad_dma_kernel<true>"),
    ((1, 8, 8, 64, 64), "wgrad_kernel<Cfg<128, 128, 2, 2>, false>"),
    ((2, 16, 32, 64, 64), "wgrad_kernel<Cfg<128, 128, 2, 2>, true>"),
]


def _closed_form(n, h, w, a):
    cr = np.array([h - 1, h, h - 1], np.float64)
    cs = np.array([w - 1, w, w - 1], np.float64)
    with np.errstate(over="ignore"):  # RNE to fp16, overflow -> +inf
        return (a * a * n * np.outer(cr, cs)).astype(np.float16)


def _run(d, x, dy, shape_w):
    ws = workspace(d, fg.OP_BWD_WEIGHT)
    plain, checked = empty16(shape_w), empty16(shape_w)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    fg.conv2d_bwd_weight(d, x, dy, plain, ws)
    fg.conv2d_bwd_weight_checked(d, x, dy, checked, flag, ws)
    return host(plain), host(checked), int(host(flag)[0])


@pytest.mark.parametrize("shape,kern", PATHS, ids=[k for _, k in PATHS])
def test_checked_kernel_gradient_closed_form(shape, kern):
    n, h, w, c, k = shape
    d = fg.ConvDesc.make(n, h, w, c, k, 3, 3, 1, 1)
    assert fg.kernel_name(d, fg.OP_BWD_WEIGHT) == kern
    a = 2.0 ** (8 - np.log2(n * h * w) / 2)  # a^2 n h w = 65536
    assert a == int(a) and a >= 1
    for scale, overflow in ((a, True), (a / 2, False)):
        ref = _closed_form(n, h, w, scale)
        assert np.isinf(ref[1, 1]) == overflow and np.isfinite(ref[[0, 0, 2, 2], [0, 2, 0, 2]]).all()
        assert np.isfinite(np.delete(ref.ravel(), 4)).all()
        x = dev(np.full((n, h, w, c), scale, np.float16))
        dy = dev(np.full((n, h, w, k), scale, np.float16))
        plain, checked, flag = _run(d, x, dy, (k, 3, 3, c))
        assert np.array_equal(plain.view(np.uint16), checked.view(np.uint16))
        for kk in (0, k // 2, k - 1):
            for cc in (0, c // 3, c - 1):
                np.testing.assert_array_equal(checked[kk, :, :, cc], ref)
        assert flag == int(overflow)


def test_checked_head_gradient():
    """K = 1 head: dW[c] = a^2 * n * h * w for constant inputs."""
    n, h, w, c = 1, 16, 16, 256
    d = fg.ConvDesc.make(n, h, w, c, 1, 1, 1, 1, 0)
    assert fg.kernel_name(d, fg.OP_BWD_WEIGHT) == "head_wgrad_kernel"
    for scale, overflow in ((16.0, True), (8.0, False)):
        x = dev(np.full((n, h, w, c), scale, np.float16))
        dy = dev(np.full((n, h, w, 1), scale, np.float16))
        plain, checked, flag = _run(d, x, dy, (1, 1, 1, c))
        assert np.array_equal(plain.view(np.uint16), checked.view(np.uint16))
        with np.errstate(over="ignore"):
            ref = np.float16(scale * scale * n * h * w)
        assert (checked.ravel() == ref).all() and flag == int(overflow)


def test_checked_random_inputs_match_plain():
    """Seeded random inputs on the split DMA path: same bits, flag 0."""
    rng = np.random.default_rng(31)
    n, h, w, c, k = 2, 45, 47, 256, 512
    d = fg.ConvDesc.make(n, h, w, c, k, 3, 3, 2, 1)
    x = dev(synth.uniform(rng, (n, h, w, c)))
    p, q = (h + 1) // 2, (w + 1) // 2
    dy = dev(synth.uniform(rng, (n, p, q, k)))
    plain, checked, flag = _run(d, x, dy, (k, 3, 3, c))
    assert np.array_equal(plain.view(np.uint16), checked.view(np.uint16)) and flag == 0


@pytest.mark.parametrize("streams", [1, 3])
def test_zero_copy_step_matches_packed_step(streams):
    """Reduced network, groups capped at 64 KiB: the zero-copy step and the
    packing step give identical master gradients, fp16 group buffers and
    flags."""
    layers = synth.fcn_layers(n=1, h=64, c_in=32, widths=(32, 64, 64, 64),
                              dec=(64, 64, 32, 32))
    x = synth.diffraction_like(1, 64, 32, seed=0)
    w = synth.he_weights(layers, seed=1)
    t = dev(synth.smooth_target(1, 64, seed=4))
    out = []
    for zc in (False, True):
        ch = Chain(layers, w, x, group_cap_bytes=64 * 1024, zero_copy=zc)
        prog = ch.program(t, streams=streams)
        prog.run()
        prog.run()  # a second step: flags are reset, slots rewritten
        torch.cuda.synchronize()
        out.append(([host(m).view(np.uint32).copy() for m in ch.master],
                    [host(g).view(np.uint16).copy() for g in ch.gbuf16],
                    host(ch.flags).copy()))
    (m0, g0, f0), (m1, g1, f1) = out
    assert all(np.array_equal(a, b) for a, b in zip(m0, m1))
    assert all(np.array_equal(a, b) for a, b in zip(g0, g1))
    np.testing.assert_array_equal(f0, f1)
    assert len(g0) > 1
