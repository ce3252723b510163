"""GPU parity of the convolution passes against the fp64 oracle.

Every case draws seeded fp16 inputs (synth), runs one library call through
the C ABI, and compares with the oracle on the same fp16 inputs under the
parity rule in gpu_util. Shapes span several tiles with ragged tails, the
generic (channels not a multiple of 64) and fast reduction paths, strides
1 and 2, 1x1 / 3x3 / 4x4 kernels, every epilogue, and the K=1 head.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1909_11150_amd as fg
import synth
from gpu_util import conv_parity, dev, empty16, host, workspace

pytestmark = pytest.mark.gpu

# n, h, w, c, k, r, stride, pad
SHAPES = [
    (2, 64, 64, 16, 16, 3, 1, 1),     # single-conv workload
    (2, 19, 23, 72, 136, 3, 1, 1),    # ragged tiles, generic reduction path
    (1, 33, 17, 64, 64, 3, 2, 1),     # stride 2, odd sizes
    (3, 12, 12, 128, 200, 1, 1, 0),   # 1x1
    (1, 16, 16, 256, 256, 3, 2, 1),   # fast path, stride 2
    (2, 9, 9, 24, 32, 4, 2, 1),       # 4x4 s2 p1 kernel (convT backward)
    (1, 7, 5, 8, 8, 3, 1, 0),         # no padding, tiny
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


def _desc(shape):
    n, h, w, c, k, r, st, pd = shape
    return fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("epi", ["none", "relu", "gate"])
def test_fwd(shape, epi):
    x, W, dy = _inputs(shape, 1)
    d = _desc(shape)
    gate = synth.uniform(np.random.default_rng(9), dy.shape) if epi == "gate" else None
    y = empty16(dy.shape)
    fg.conv2d_fwd(d, dev(x), dev(W), y, {"none": 0, "relu": 1, "gate": 2}[epi],
                  dev(gate) if gate is not None else None, workspace(d, fg.OP_FWD))
    ref = oracle.conv2d_fwd(x, W, shape[6], shape[7],
                            epi=None if epi == "none" else epi, gate=gate)
    conv_parity(host(y), ref, f"fwd {shape} {epi}")


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("epi", ["none", "gate"])
def test_bwd_data(shape, epi):
    x, W, dy = _inputs(shape, 2)
    d = _desc(shape)
    gate = synth.uniform(np.random.default_rng(8), x.shape) if epi == "gate" else None
    dx = empty16(x.shape)
    fg.conv2d_bwd_data(d, dev(dy), dev(W), dx, 2 if epi == "gate" else 0,
                       dev(gate) if gate is not None else None,
                       workspace(d, fg.OP_BWD_DATA))
    ref = oracle.conv2d_bwd_data(dy, W, x.shape, shape[6], shape[7],
                                 epi=None if epi == "none" else epi, gate=gate)
    conv_parity(host(dx), ref, f"bwd_data {shape} {epi}")


@pytest.mark.parametrize("shape", SHAPES)
def test_bwd_weight(shape):
    x, W, dy = _inputs(shape, 3)
    d = _desc(shape)
    dw = empty16(W.shape)
    fg.conv2d_bwd_weight(d, dev(x), dev(dy), dw, workspace(d, fg.OP_BWD_WEIGHT))
    ref = oracle.conv2d_bwd_weight(x, dy, shape[5], shape[5], shape[6], shape[7])
    conv_parity(host(dw), ref, f"bwd_weight {shape}")


CONVT = [(1, 5, 7, 16, 24), (2, 8, 8, 64, 128), (1, 32, 32, 256, 128),
         (3, 1, 1, 8, 8)]


@pytest.mark.parametrize("shape", CONVT)
@pytest.mark.parametrize("epi", ["none", "relu", "gate"])
def test_convt(shape, epi):
    n, h, w, ci, co = shape
    rng = np.random.default_rng(4)
    x = synth.uniform(rng, (n, h, w, ci))
    Wt = synth.normal(rng, (ci, 4, 4, co), np.sqrt(2.0 / (4 * ci)))
    oshape = (n, 2 * h, 2 * w, co)
    gate = synth.uniform(rng, oshape) if epi == "gate" else None
    y = empty16(oshape)
    d = fg.ConvDesc.make(n, h, w, ci, co, 4, 4, 2, 1)
    fg.conv_transpose2d_fwd(d, dev(x), dev(Wt), y,
                            {"none": 0, "relu": 1, "gate": 2}[epi],
                            dev(gate) if gate is not None else None,
                            workspace(d, fg.OP_CONVT))
    ref = oracle.conv_transpose2d_fwd(x, Wt, 2, 1,
                                      epi=None if epi == "none" else epi, gate=gate)
    conv_parity(host(y), ref, f"convT {shape} {epi}")


def test_convt_matches_bwd_data_with_roles_exchanged():
    """conv_transpose2d_fwd(x; Wt) and conv2d_bwd_data(dy := x; W := Wt)
    evaluate the same operator."""
    rng = np.random.default_rng(5)
    x = synth.uniform(rng, (2, 8, 8, 64))
    Wt = synth.normal(rng, (64, 4, 4, 32), 0.05)
    y1, y2 = empty16((2, 16, 16, 32)), empty16((2, 16, 16, 32))
    dt = fg.ConvDesc.make(2, 8, 8, 64, 32, 4, 4, 2, 1)
    db = fg.ConvDesc.make(2, 16, 16, 32, 64, 4, 4, 2, 1)
    fg.conv_transpose2d_fwd(dt, dev(x), dev(Wt), y1, ws=workspace(dt, fg.OP_CONVT))
    fg.conv2d_bwd_data(db, dev(x), dev(Wt), y2, ws=workspace(db, fg.OP_BWD_DATA))
    np.testing.assert_array_equal(host(y1), host(y2))


@pytest.mark.parametrize("npix_hw", [(4, 256, 256), (1, 7, 9)])
@pytest.mark.parametrize("c", [256, 24])
def test_head_k1(npix_hw, c):
    """The single-output-channel 1x1 head: all three passes."""
    n, h, w = npix_hw
    rng = np.random.default_rng(6)
    x = np.maximum(synth.uniform(rng, (n, h, w, c)), np.float16(0))
    W = synth.normal(rng, (1, 1, 1, c), np.sqrt(2.0 / c))
    dy = synth.uniform(rng, (n, h, w, 1))
    d = fg.ConvDesc.make(n, h, w, c, 1, 1, 1, 1, 0)
    y = empty16((n, h, w, 1))
    fg.conv2d_fwd(d, dev(x), dev(W), y)
    conv_parity(host(y), oracle.conv2d_fwd(x, W, 1, 0), "head fwd")
    dx = empty16(x.shape)
    fg.conv2d_bwd_data(d, dev(dy), dev(W), dx, fg.EPI_GATE, dev(x))
    ref = oracle.conv2d_bwd_data(dy, W, x.shape, 1, 0, epi="gate", gate=x)
    # one product per output: exact up to the single fp16 rounding
    np.testing.assert_array_equal(host(dx), ref.astype(np.float16))
    ws = torch.empty(fg.workspace_bytes(d, fg.OP_BWD_WEIGHT), dtype=torch.uint8,
                     device="cuda")
    dw = empty16(W.shape)
    fg.conv2d_bwd_weight(d, dev(x), dev(dy), dw, ws)
    conv_parity(host(dw), oracle.conv2d_bwd_weight(x, dy, 1, 1, 1, 0), "head dW")


def test_identity_weight_is_bit_exact():
    """A 1x1 identity kernel reproduces x exactly (one nonzero product)."""
    rng = np.random.default_rng(7)
    x = synth.uniform(rng, (2, 10, 11, 64))
    eye = np.eye(64, dtype=np.float16).reshape(64, 1, 1, 64)
    y = empty16(x.shape)
    d = fg.ConvDesc.make(2, 10, 11, 64, 64, 1, 1, 1, 0)
    fg.conv2d_fwd(d, dev(x), dev(eye), y, ws=workspace(d, fg.OP_FWD))
    np.testing.assert_array_equal(host(y), x)


def test_all_ones_weight_gradient_rounds_to_even():
    """x = dy = 1 on the single-conv shape: dW = 2*cnt(r)*cnt(s) with counts
    (63, 64, 63); 7938 is a tie between fp16 neighbours and must give 7936."""
    x = np.ones((2, 64, 64, 16), np.float16)
    dy = np.ones((2, 64, 64, 16), np.float16)
    d = fg.ConvDesc.make(2, 64, 64, 16, 16, 3, 3, 1, 1)
    dw = empty16((16, 3, 3, 16))
    fg.conv2d_bwd_weight(d, dev(x), dev(dy), dw, workspace(d, fg.OP_BWD_WEIGHT))
    got = host(dw)
    cnt = np.array([63, 64, 63])
    ref = (2 * np.outer(cnt, cnt)).astype(np.float16)
    for k in (0, 7, 15):
        for c in (0, 9, 15):
            np.testing.assert_array_equal(got[k, :, :, c], ref)
    assert got[0, 0, 0, 0] == 7936


def test_fp16_overflow_gives_infinity():
    """Outputs beyond the fp16 range become exactly +-inf (no saturation)."""
    x = np.full((1, 4, 4, 64), 60.0, np.float16)
    W = np.full((8, 1, 1, 64), 30.0, np.float16)
    W[1::2] *= -1
    y = empty16((1, 4, 4, 8))
    d = fg.ConvDesc.make(1, 4, 4, 64, 8, 1, 1, 1, 0)
    fg.conv2d_fwd(d, dev(x), dev(W), y, ws=workspace(d, fg.OP_FWD))
    got = host(y)
    assert np.all(np.isposinf(got[..., 0::2])) and np.all(np.isneginf(got[..., 1::2]))


def test_adjoint_identity_on_gpu_outputs():
    """<fwd(x), dy> = <x, bwd_data(dy)> with both sides from GPU outputs."""
    shape = (2, 32, 32, 64, 128, 3, 2, 1)
    x, W, dy = _inputs(shape, 10)
    d = _desc(shape)
    y, dx = empty16(dy.shape), empty16(x.shape)
    fg.conv2d_fwd(d, dev(x), dev(W), y, ws=workspace(d, fg.OP_FWD))
    fg.conv2d_bwd_data(d, dev(dy), dev(W), dx, ws=workspace(d, fg.OP_BWD_DATA))
    lhs = float(np.sum(host(y).astype(np.float64) * dy))
    rhs = float(np.sum(x.astype(np.float64) * host(dx)))
    assert abs(lhs - rhs) <= 1e-3 * np.sqrt(np.sum(host(y).astype(np.float64) ** 2) *
                                            np.sum(dy.astype(np.float64) ** 2))


def test_deterministic_repeats():
    shape = (2, 32, 32, 128, 128, 3, 1, 1)
    x, W, dy = _inputs(shape, 11)
    d = _desc(shape)
    xs, Ws, dys = dev(x), dev(W), dev(dy)
    ws = [workspace(d, op) for op in (fg.OP_FWD, fg.OP_BWD_DATA, fg.OP_BWD_WEIGHT)]
    outs = []
    for _ in range(2):
        y, dx, dw = empty16(dy.shape), empty16(x.shape), empty16(W.shape)
        fg.conv2d_fwd(d, xs, Ws, y, ws=ws[0])
        fg.conv2d_bwd_data(d, dys, Ws, dx, ws=ws[1])
        fg.conv2d_bwd_weight(d, xs, dys, dw, ws[2])
        outs.append([host(t) for t in (y, dx, dw)])
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
