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
