"""GPU parity of strided outputs and the accumulate epilogue (the layout a
dense block's concatenation and its gradient sums need, Section 6.2).

For each output path of the data convolutions (staged 256 x 256 store with
and without a split, the input-reuse kernel, 128 x 128 tiles, the
register-staged kernel, a strided input gradient's four phases, the
transposed convolution), the pass writes into a channel slice of a wider
buffer (pixel stride = channels + 24, slice at channel 8):
  * plain: the slice equals the dense call's output bit for bit, and every
    other channel of the buffer keeps its bits;
  * FG_EPI_ACC: the slice holds fp16(old + result). The dense call's fp16
    output r16 is the fp32 result rounded, so the slice lies within half an
    ulp of r16 plus half an ulp of itself from r16 + old (the staged store
    rounds the result first, the other paths add the fp32 result); and it
    meets the single-op rule against the fp64 oracle of old + the
    convolution on sampled elements;
  * a gate laid out like the strided output (FG_EPI_GATE).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1909_11150_amd as fg
import synth
from gpu_util import conv_parity, dev, host, sample_indices, workspace

pytestmark = pytest.mark.gpu

PAD, OFF = 24, 8

# (n, h, w, c, k, r, stride, pad), op, kernel-name fragment
CASES = [
    ((2, 93, 95, 256, 512, 1, 1, 0), fg.OP_FWD, "data_conv_dma_kernel<true, false>"),
    ((1, 77, 79, 512, 512, 3, 1, 1), fg.OP_FWD, "data_conv_dma_kernel<true, true>"),
    ((2, 128, 128, 512, 320, 3, 1, 1), fg.OP_BWD_DATA, "halo"),
    ((1, 64, 64, 1024, 1024, 3, 1, 1), fg.OP_FWD, "halo"),
    ((2, 15, 17, 1024, 1024, 3, 1, 1), fg.OP_FWD, "data_conv_dma_kernel<128"),
    ((2, 16, 16, 24, 40, 3, 1, 1), fg.OP_FWD, "data_conv_kernel<"),
    ((1, 127, 129, 512, 256, 3, 2, 1), fg.OP_BWD_DATA, "data_conv_dma_kernel<false"),
    ((1, 33, 31, 1024, 512, 3, 2, 1), fg.OP_BWD_DATA, "data_conv_dma_kernel<128"),
]


def _ulp16(a):
    """Spacing of fp16 numbers at each |a| (2^-24 below the normal range)."""
    a = np.abs(np.asarray(a, np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -14)))
    return 2.0 ** (e - 10)


def _run(op, d, x, w, dy, out, epi, gate=None):
    ws = workspace(d, op)
    if op == fg.OP_FWD:
        fg.conv2d_fwd(d, x, w, out, epi, gate, ws)
    elif op == fg.OP_BWD_DATA:
        fg.conv2d_bwd_data(d, dy, w, out, epi, gate, ws)
    else:
        fg.conv_transpose2d_fwd(d, x, w, out, epi, gate, ws)


@pytest.mark.parametrize("shape,op,frag", CASES, ids=[f"{f}-{s}" for s, _, f in CASES])
def test_strided_output_and_accumulate(shape, op, frag):
    n, h, w, c, k, r, st, pd = shape
    rng = np.random.default_rng(h * w + c + k)
    p = (h + 2 * pd - r) // st + 1
    q = (w + 2 * pd - r) // st + 1
    x = synth.uniform(rng, (n, h, w, c))
    W = synth.normal(rng, (k, r, r, c), np.sqrt(2.0 / (r * r * c)))
    dy = synth.uniform(rng, (n, p, q, k))
    oshape = (n, p, q, k) if op == fg.OP_FWD else (n, h, w, c)
    ch = oshape[3]
    ld = ch + PAD
    if op == fg.OP_FWD:
        d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd, y_ld=ld)
        dd = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
    else:
        d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd, x_ld=ld)
        dd = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
    assert frag in fg.kernel_name(d, op)
    xs, Ws, dys = dev(x), dev(W), dev(dy)
    npix = int(np.prod(oshape[:3]))
    dense = torch.empty(oshape, dtype=torch.float16, device="cuda")
    _run(op, dd, xs, Ws, dys, dense, fg.EPI_NONE)
    ref16 = host(dense).reshape(npix, ch)
    old = synth.normal(rng, (npix, ld))
    for epi in (fg.EPI_NONE, fg.EPI_ACC):
        big = dev(old)
        sl = big.view(-1)[OFF:]          # the slice's first element
        _run(op, d, xs, Ws, dys, sl, epi)
        got = host(big)
        keep = np.ones(ld, bool)
        keep[OFF:OFF + ch] = False
        np.testing.assert_array_equal(got[:, keep].view(np.uint16),
                                      old[:, keep].view(np.uint16))
        g = got[:, OFF:OFF + ch]
        if epi == fg.EPI_NONE:
            np.testing.assert_array_equal(g.view(np.uint16), ref16.view(np.uint16))
            continue
        o = old[:, OFF:OFF + ch]
        err = np.abs(g.astype(np.float64) - (ref16.astype(np.float64) + o.astype(np.float64)))
        bound = 0.5 * _ulp16(ref16) + 0.5 * _ulp16(g)
        assert np.all(err <= bound), float((err / bound).max())
        idx = sample_indices(oshape, 1500, rng)
        if op == fg.OP_FWD:
            conv = oracle.conv2d_fwd_points(x, W, idx, st, pd)
        else:
            conv = oracle.conv2d_bwd_data_points(dy, W, x.shape, idx, st, pd)
        conv_parity(g.ravel()[idx], conv + o.ravel()[idx].astype(np.float64), "acc")


def test_strided_convt_and_gate():
    n, h, w, ci, co = 1, 65, 66, 256, 512
    rng = np.random.default_rng(5)
    x = synth.uniform(rng, (n, h, w, ci))
    Wt = synth.normal(rng, (ci, 4, 4, co), np.sqrt(2.0 / (4 * ci)))
    oshape = (n, 2 * h, 2 * w, co)
    npix = int(np.prod(oshape[:3]))
    ld = co + PAD
    d = fg.ConvDesc.make(n, h, w, ci, co, 4, 4, 2, 1, y_ld=ld)
    dd = fg.ConvDesc.make(n, h, w, ci, co, 4, 4, 2, 1)
    dense = torch.empty(oshape, dtype=torch.float16, device="cuda")
    gate = synth.normal(rng, (npix, ld))
    fg.conv_transpose2d_fwd(dd, dev(x), dev(Wt), dense, fg.EPI_GATE,
                            dev(np.ascontiguousarray(gate[:, OFF:OFF + co])),
                            workspace(dd, fg.OP_CONVT))
    big = torch.zeros((npix, ld), dtype=torch.float16, device="cuda")
    fg.conv_transpose2d_fwd(d, dev(x), dev(Wt), big.view(-1)[OFF:], fg.EPI_GATE,
                            dev(gate).view(-1)[OFF:], workspace(d, fg.OP_CONVT))
    got = host(big)
    np.testing.assert_array_equal(got[:, OFF:OFF + co].view(np.uint16),
                                  host(dense).reshape(npix, co).view(np.uint16))
    assert not np.any(got[:, :OFF]) and not np.any(got[:, OFF + co:])


# strided inputs: the forward pass and the kernel gradient reading x from a
# channel slice of a wider buffer, on each kernel path
IN_CASES = [(s, f) for s, op, f in CASES if op == fg.OP_FWD] + \
    [((1, 127, 129, 512, 256, 3, 2, 1), "")]
WG_FRAGS = ("wgrad_dma_kernel<false>", "wgrad_dma_kernel<true>", "wgrad_kernel<")


@pytest.mark.parametrize("shape,frag", IN_CASES, ids=[f"{f}-{s}" for s, f in IN_CASES])
def test_strided_input(shape, frag):
    """x at channel OFF of a buffer of pixel stride c + PAD: the forward
    output (with ReLU) and the kernel gradient equal the dense calls' bit
    for bit, and the buffer is left as it was."""
    n, h, w, c, k, r, st, pd = shape
    rng = np.random.default_rng(h * w + c + k + 1)
    p = (h + 2 * pd - r) // st + 1
    q = (w + 2 * pd - r) // st + 1
    x = synth.uniform(rng, (n, h, w, c))
    W = synth.normal(rng, (k, r, r, c), np.sqrt(2.0 / (r * r * c)))
    dy = synth.uniform(rng, (n, p, q, k))
    ld = c + PAD
    npx = n * h * w
    big = synth.normal(rng, (npx, ld))
    big[:, OFF:OFF + c] = x.reshape(npx, c)
    bigd = dev(big)
    xs = bigd.view(-1)[OFF:]
    dd = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
    ds = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd, x_ld=ld)
    assert frag in fg.kernel_name(ds, fg.OP_FWD)
    print(fg.kernel_name(ds, fg.OP_FWD), fg.kernel_name(ds, fg.OP_BWD_WEIGHT))
    Ws, dys, xd = dev(W), dev(dy), dev(x)
    ys = [torch.empty((n, p, q, k), dtype=torch.float16, device="cuda") for _ in range(2)]
    dws = [torch.empty((k, r, r, c), dtype=torch.float16, device="cuda") for _ in range(2)]
    for d, xx, y, dw in ((dd, xd, ys[0], dws[0]), (ds, xs, ys[1], dws[1])):
        fg.conv2d_fwd(d, xx, Ws, y, fg.EPI_RELU, None, workspace(d, fg.OP_FWD))
        fg.conv2d_bwd_weight(d, xx, dys, dw, workspace(d, fg.OP_BWD_WEIGHT))
    np.testing.assert_array_equal(host(ys[1]).view(np.uint16), host(ys[0]).view(np.uint16))
    np.testing.assert_array_equal(host(dws[1]).view(np.uint16), host(dws[0]).view(np.uint16))
    np.testing.assert_array_equal(host(bigd).view(np.uint16), big.view(np.uint16))


def test_strided_kernel_gradient_paths_covered():
    names = {fg.kernel_name(fg.ConvDesc.make(*s, x_ld=s[3] + PAD), fg.OP_BWD_WEIGHT)
             for s, _ in IN_CASES}
    for f in WG_FRAGS:
        assert any(f in nm for nm in names), (f, names)


def test_interleaved_input_and_output():
    """A dense block's layer: x = channels [0, c) of a buffer, the output
    written (then added, FG_EPI_ACC) into channels [c, c + k) of the same
    buffer at the same pixel stride."""
    n, h, w, c, k = 2, 64, 64, 256, 256
    rng = np.random.default_rng(17)
    ld = c + k + 8
    npx = n * h * w
    big = synth.normal(rng, (npx, ld))
    x = np.ascontiguousarray(big[:, :c]).reshape(n, h, w, c)
    W = synth.normal(rng, (k, 3, 3, c), np.sqrt(2.0 / (9 * c)))
    dd = fg.ConvDesc.make(n, h, w, c, k, 3, 3, 1, 1)
    ds = fg.ConvDesc.make(n, h, w, c, k, 3, 3, 1, 1, x_ld=ld, y_ld=ld)
    Ws = dev(W)
    ref = torch.empty((n, h, w, k), dtype=torch.float16, device="cuda")
    fg.conv2d_fwd(dd, dev(x), Ws, ref, fg.EPI_NONE, None, workspace(dd, fg.OP_FWD))
    r16 = host(ref).reshape(npx, k)
    bigd = dev(big)
    fg.conv2d_fwd(ds, bigd, Ws, bigd.view(-1)[c:], fg.EPI_NONE, None,
                  workspace(ds, fg.OP_FWD))
    got = host(bigd)
    np.testing.assert_array_equal(got[:, c:c + k].view(np.uint16), r16.view(np.uint16))
    keep = np.ones(ld, bool)
    keep[c:c + k] = False
    np.testing.assert_array_equal(got[:, keep].view(np.uint16), big[:, keep].view(np.uint16))
    fg.conv2d_fwd(ds, bigd, Ws, bigd.view(-1)[c:], fg.EPI_ACC, None,
                  workspace(ds, fg.OP_FWD))
    g = host(bigd)[:, c:c + k].astype(np.float64)
    err = np.abs(g - 2.0 * r16.astype(np.float64))
    assert np.all(err <= 0.5 * _ulp16(2.0 * r16) + 0.5 * _ulp16(g)), float(err.max())
