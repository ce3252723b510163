"""GPU parity of the input-reuse ("halo") kernel for stride-1 3x3 convolutions.

Stride-1 3x3 forward and input-gradient passes whose 256-position output
tile is a block of whole output rows go to a kernel that loads each tile's
input window (with a one-pixel halo) once per 32-channel chunk and reads the
nine taps as shifted views of it. The cases below reach it with image widths
16 to 128, output channels that do not fill the last tile, zero padding at
every border, several images per batch and split reductions; outputs are
checked on sampled elements (plus all corners) against the oracle.
"""
import numpy as np
import pytest

import oracle
import paper_1909_11150_amd as fg
import synth
from gpu_util import conv_parity, dev, empty16, host, sample_indices, workspace

pytestmark = pytest.mark.gpu

# (n, h, w, c, k), op
CASES = [
    ((1, 64, 64, 1024, 1024), fg.OP_FWD),      # split reduction, width 64
    ((4, 32, 32, 1024, 1024), fg.OP_FWD),      # width 32, 4 images per batch
    ((2, 128, 128, 256, 320), fg.OP_FWD),      # width 128, ragged channel tile
    ((2, 64, 128, 1024, 256), fg.OP_FWD),
    ((1, 64, 64, 1024, 1024), fg.OP_BWD_DATA),
    ((4, 32, 32, 1024, 1024), fg.OP_BWD_DATA),
    ((2, 128, 128, 512, 320), fg.OP_BWD_DATA),  # 10 channel chunks
    ((1, 128, 128, 1024, 256), fg.OP_BWD_DATA),
]


def _inputs(shape, seed):
    n, h, w, c, k = shape
    rng = np.random.default_rng(seed)
    x = np.maximum(synth.uniform(rng, (n, h, w, c)), np.float16(0))
    W = synth.normal(rng, (k, 3, 3, c), np.sqrt(2.0 / (9 * c)))
    dy = synth.uniform(rng, (n, h, w, k))
    return x, W, dy


@pytest.mark.parametrize("shape,op", CASES,
                         ids=[f"{'fwd' if o == fg.OP_FWD else 'dx'}-{s}" for s, o in CASES])
def test_halo_conv(shape, op):
    n, h, w, c, k = shape
    d = fg.ConvDesc.make(n, h, w, c, k, 3, 3, 1, 1)
    assert fg.kernel_name(d, op).startswith("data_conv_halo_kernel<")
    x, W, dy = _inputs(shape, 31)
    rng = np.random.default_rng(32)
    ws = workspace(d, op)
    if op == fg.OP_FWD:
        y = empty16(dy.shape)
        fg.conv2d_fwd(d, dev(x), dev(W), y, fg.EPI_RELU, None, ws)
        idx = sample_indices(dy.shape, 3000, rng)
        ref = oracle.relu(oracle.conv2d_fwd_points(x, W, idx, 1, 1))
        conv_parity(host(y).ravel()[idx], ref, f"fwd {shape}")
    else:
        dx = empty16(x.shape)
        fg.conv2d_bwd_data(d, dev(dy), dev(W), dx, fg.EPI_GATE, dev(x), ws)
        idx = sample_indices(x.shape, 3000, rng)
        ref = oracle.conv2d_bwd_data_points(dy, W, x.shape, idx, 1, 1)
        ref = np.where(x.ravel()[idx].astype(np.float64) > 0, ref, 0.0)
        conv_parity(host(dx).ravel()[idx], ref, f"dx {shape}")


def test_halo_variants_reached():
    """Both the split and the unsplit kernels are among the cases above."""
    names = {fg.kernel_name(fg.ConvDesc.make(*s, 3, 3, 1, 1), o) for s, o in CASES}
    assert any(nm.endswith("true>") for nm in names)
    assert any(nm.endswith("false>") for nm in names)


def test_halo_deterministic():
    shape = (2, 128, 128, 256, 320)
    n, h, w, c, k = shape
    d = fg.ConvDesc.make(n, h, w, c, k, 3, 3, 1, 1)
    x, W, dy = _inputs(shape, 33)
    xs, Ws = dev(x), dev(W)
    outs = []
    for _ in range(2):
        y = empty16(dy.shape)
        fg.conv2d_fwd(d, xs, Ws, y, fg.EPI_NONE, None, workspace(d, fg.OP_FWD))
        outs.append(host(y).view(np.uint16).copy())
    assert np.array_equal(outs[0], outs[1])
