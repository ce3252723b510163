"""GPU parity of the LDS-DMA kernels on ragged shapes.

The tile planner sends large shapes to the LDS-DMA kernels (256 x 256
tiles fed by buffer loads straight into LDS) and shapes with few output
positions to their 128 x 128 version. These cases are chosen so that
each of those kernels is reached with ragged edges: output positions and
channels that do not fill the last tile, odd image sizes with padding at the
borders, stride-2 phases, reduction splits and partial last stages. Outputs
are checked on sampled elements (plus all corners) against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1909_11150_amd as fg
import synth
from gpu_util import conv_parity, dev, empty16, host, sample_indices, workspace

pytestmark = pytest.mark.gpu

# (n, h, w, c, k, r, stride, pad), op, expected kernel
CASES = [
    ((2, 93, 95, 256, 512, 1, 1, 0), fg.OP_FWD, "data_conv_dma_kernel<true, false>"),
    ((1, 77, 79, 512, 512, 3, 1, 1), fg.OP_FWD, "data_conv_dma_kernel<true, true>"),
    ((4, 77, 79, 288, 256, 1, 1, 0), fg.OP_BWD_DATA, "data_conv_dma_kernel<false, false>"),
    ((1, 77, 79, 512, 512, 3, 1, 1), fg.OP_BWD_DATA, "data_conv_dma_kernel<false, true>"),
    ((1, 127, 129, 512, 256, 3, 2, 1), fg.OP_BWD_DATA, "data_conv_dma_kernel<false, false>"),
    ((1, 93, 95, 512, 512, 3, 1, 1), fg.OP_BWD_WEIGHT, "wgrad_dma_kernel<true>"),
    # 128 x 128 tiles
    ((2, 15, 17, 1024, 1024, 3, 1, 1), fg.OP_FWD, "data_conv_dma_kernel<128, true, true>"),
    ((8, 64, 64, 64, 128, 3, 1, 1), fg.OP_FWD, "data_conv_dma_kernel<128, true, false>"),
    ((1, 31, 33, 512, 768, 3, 2, 1), fg.OP_FWD, "data_conv_dma_kernel<128, true, true>"),
    ((4, 64, 64, 256, 128, 3, 1, 1), fg.OP_BWD_DATA, "data_conv_dma_kernel<128, false, false>"),
    ((1, 33, 31, 1024, 512, 3, 2, 1), fg.OP_BWD_DATA, "data_conv_dma_kernel<128, false, true>"),
]


def _inputs(shape, seed):
    n, h, w, c, k, r, st, pd = shape
    rng = np.random.default_rng(seed)
    p = (h + 2 * pd - r) // st + 1
    q = (w + 2 * pd - r) // st + 1
    x = synth.uniform(rng, (n, h, w, c))
    W = synth.normal(rng, (k, r, r, c), np.sqrt(2.0 / (r * r * c)))
    dy = synth.uniform(rng, (n, p, q, k))
    return x, W, dy


@pytest.mark.parametrize("shape,op,kern", CASES,
                         ids=[f"{k}-{s}" for s, _, k in CASES])
def test_dma_conv(shape, op, kern):
    n, h, w, c, k, r, st, pd = shape
    d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
    assert fg.kernel_name(d, op) == kern
    x, W, dy = _inputs(shape, 21)
    rng = np.random.default_rng(22)
    ws = workspace(d, op)
    if op == fg.OP_FWD:
        y = empty16(dy.shape)
        fg.conv2d_fwd(d, dev(x), dev(W), y, fg.EPI_RELU, None, ws)
        idx = sample_indices(dy.shape, 3000, rng)
        ref = oracle.relu(oracle.conv2d_fwd_points(x, W, idx, st, pd))
        conv_parity(host(y).ravel()[idx], ref, f"fwd {shape}")
    elif op == fg.OP_BWD_DATA:
        dx = empty16(x.shape)
        fg.conv2d_bwd_data(d, dev(dy), dev(W), dx, fg.EPI_GATE, dev(x), ws)
        idx = sample_indices(x.shape, 3000, rng)
        ref = oracle.conv2d_bwd_data_points(dy, W, x.shape, idx, st, pd)
        ref = np.where(x.ravel()[idx].astype(np.float64) > 0, ref, 0.0)
        conv_parity(host(dx).ravel()[idx], ref, f"dx {shape}")
    else:
        dw = empty16(W.shape)
        fg.conv2d_bwd_weight(d, dev(x), dev(dy), dw, ws)
        idx = sample_indices(W.shape, 2000, rng)
        ref = oracle.conv2d_bwd_weight_points(x, dy, r, r, idx, st, pd)
        conv_parity(host(dw).ravel()[idx], ref, f"dW {shape}")


def test_dma_convt_ragged():
    n, h, w, ci, co = 1, 65, 66, 256, 512
    d = fg.ConvDesc.make(n, h, w, ci, co, 4, 4, 2, 1)
    assert fg.kernel_name(d, fg.OP_CONVT) == "data_conv_dma_kernel<false, false>"
    rng = np.random.default_rng(23)
    x = synth.uniform(rng, (n, h, w, ci))
    Wt = synth.normal(rng, (ci, 4, 4, co), np.sqrt(2.0 / (4 * ci)))
    y = empty16((n, 2 * h, 2 * w, co))
    fg.conv_transpose2d_fwd(d, dev(x), dev(Wt), y, fg.EPI_NONE, None,
                            workspace(d, fg.OP_CONVT))
    idx = sample_indices(y.shape, 3000, rng)
    ref = oracle.conv_transpose2d_fwd_points(x, Wt, idx, 2, 1)
    conv_parity(host(y).ravel()[idx], ref, "convT")


def test_dma_small_convt_ragged():
    n, h, w, ci, co = 1, 15, 16, 1024, 1024
    d = fg.ConvDesc.make(n, h, w, ci, co, 4, 4, 2, 1)
    assert fg.kernel_name(d, fg.OP_CONVT) == "data_conv_dma_kernel<128, false, true>"
    rng = np.random.default_rng(25)
    x = synth.uniform(rng, (n, h, w, ci))
    Wt = synth.normal(rng, (ci, 4, 4, co), np.sqrt(2.0 / (4 * ci)))
    y = empty16((n, 2 * h, 2 * w, co))
    fg.conv_transpose2d_fwd(d, dev(x), dev(Wt), y, fg.EPI_RELU, None,
                            workspace(d, fg.OP_CONVT))
    idx = sample_indices(y.shape, 3000, rng)
    ref = oracle.relu(oracle.conv_transpose2d_fwd_points(x, Wt, idx, 2, 1))
    conv_parity(host(y).ravel()[idx], ref, "convT small")


def test_dma_deterministic():
    """Two runs of a DMA-kernel convolution give identical bits."""
    shape = (2, 93, 95, 256, 512, 1, 1, 0)
    n, h, w, c, k, r, st, pd = shape
    d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
    x, W, dy = _inputs(shape, 24)
    xs, Ws = dev(x), dev(W)
    outs = []
    for _ in range(2):
        y = empty16(dy.shape)
        fg.conv2d_fwd(d, xs, Ws, y, fg.EPI_NONE, None, workspace(d, fg.OP_FWD))
        outs.append(host(y).view(np.uint16).copy())
    assert np.array_equal(outs[0], outs[1])
