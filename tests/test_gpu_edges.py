"""fp16 range edges on every convolution kernel path: outputs that overflow
to +-inf and outputs in the subnormal range (Section 6.2: float16 training
with loss scaling; fp16 conversions round to nearest-even, overflow to
infinity, and keep subnormals).

Each case names the kernel the planner must pick for it, and runs two input
recipes whose every partial sum is exact in fp32, so that the fp64 oracle
value rounded once to fp16 is the exact answer and the GPU must match it
value for value (+0 and -0 compare equal), whatever the accumulation order
or the split of the reduction:

  overflow   the data operand is +-2^e per pixel (e in 0..3, the same for
             all channels; per element for the kernel gradient, whose sums
             run over pixels) and the other operand depends only on the output
             channel: +-b * 2^(j mod 2). Every term is an integer multiple
             of b of magnitude at most 16 b, and no output sums more than
             2^18 terms, so every partial sum is exact in fp32; b, a power
             of two, puts the outputs around the fp16 overflow threshold, so
             some reach +-inf and some stay finite.
  subnormal  data and convolutions: data values m * 2^-24 (|m| in
             1..1023) and a delta kernel at one tap; the outputs are
             single values or sums of a few, all multiples of 2^-24.
             Kernel gradients: one nonzero pixel per image (2^-12 * {1, 2,
             3}) against an output gradient of +-2^-8 * {1, 2}, so each dW
             is a sum of at most N products of size 2^-20 * {1 .. 6}.
"""
import numpy as np
import pytest

import oracle
import paper_1909_11150_amd as fg
from gpu_util import dev, empty16, host, sample_indices, workspace

pytestmark = pytest.mark.gpu

FWD, DX, DW = fg.OP_FWD, fg.OP_BWD_DATA, fg.OP_BWD_WEIGHT

# (n, h, w, c, k, r, stride, pad), op, the kernel the planner picks
CASES = [
    ((2, 93, 95, 256, 512, 1, 1, 0), FWD, "data_conv_dma_kernel<true, false>"),
    ((1, 77, 79, 512, 512, 3, 1, 1), FWD, "data_conv_dma_kernel<true, true>"),
    ((8, 64, 64, 64, 128, 3, 1, 1), FWD, "data_conv_dma_kernel<128, true, false>"),
    ((2, 15, 17, 1024, 1024, 3, 1, 1), FWD, "data_conv_dma_kernel<128, true, true>"),
    ((1, 127, 129, 512, 256, 3, 2, 1), FWD, "data_conv_dma_kernel<128, true, true>"),
    ((2, 128, 128, 256, 320, 3, 1, 1), FWD, "data_conv_halo_kernel<true, false>"),
    ((1, 64, 64, 1024, 1024, 3, 1, 1), FWD, "data_conv_halo_kernel<true, true>"),
    ((2, 64, 64, 16, 16, 3, 1, 1), FWD,
     "data_conv_kernel<Cfg<128, 128, 2, 2>, true, false, false>"),
    ((2, 20, 21, 48, 40, 3, 2, 1), FWD,
     "data_conv_kernel<Cfg<128, 128, 2, 2>, true, false, true>"),
    ((4, 128, 128, 264, 512, 3, 1, 1), FWD,
     "data_conv_kernel<Cfg<256, 256, 2, 4>, true, false, false>"),
    ((2, 30, 30, 64, 1, 1, 1, 0), FWD, "head_fwd_kernel"),
    ((4, 77, 79, 288, 256, 1, 1, 0), DX, "data_conv_dma_kernel<false, false>"),
    ((1, 127, 129, 512, 256, 3, 2, 1), DX, "data_conv_dma_kernel<false, false>"),
    ((1, 77, 79, 512, 512, 3, 1, 1), DX, "data_conv_dma_kernel<false, true>"),
    ((4, 64, 64, 256, 128, 3, 1, 1), DX, "data_conv_dma_kernel<128, false, false>"),
    ((1, 33, 31, 1024, 512, 3, 2, 1), DX, "data_conv_dma_kernel<128, false, true>"),
    ((2, 128, 128, 512, 320, 3, 1, 1), DX, "data_conv_halo_kernel<false, false>"),
    ((1, 64, 64, 1024, 1024, 3, 1, 1), DX, "data_conv_halo_kernel<false, true>"),
    ((2, 20, 21, 48, 40, 3, 2, 1), DX,
     "data_conv_kernel<Cfg<128, 128, 2, 2>, false, false, false>"),
    ((2, 20, 21, 40, 48, 3, 1, 1), DX,
     "data_conv_kernel<Cfg<128, 128, 2, 2>, false, false, true>"),
    ((4, 128, 128, 512, 264, 3, 1, 1), DX,
     "data_conv_kernel<Cfg<256, 256, 2, 4>, false, false, false>"),
    ((2, 30, 30, 64, 1, 1, 1, 0), DX, "head_bwd_data_kernel"),
    ((1, 77, 79, 512, 512, 3, 1, 1), DW, "wgrad_dma_kernel<true>"),
    ((2, 15, 17, 1024, 1024, 3, 1, 1), DW, "wgrad_dma_kernel<false>"),
    ((2, 20, 21, 48, 40, 3, 2, 1), DW, "wgrad_kernel<Cfg<128, 128, 2, 2>, false>"),
    ((2, 64, 64, 16, 16, 3, 1, 1), DW, "wgrad_kernel<Cfg<128, 128, 2, 2>, true>"),
    ((1, 64, 64, 264, 512, 3, 2, 1), DW, "wgrad_kernel<Cfg<256, 256, 2, 4>, false>"),
    ((4, 77, 79, 288, 256, 1, 1, 0), DW, "wgrad_kernel<Cfg<256, 256, 2, 4>, true>"),
    ((2, 30, 30, 64, 1, 1, 1, 0), DW, "head_wgrad_kernel"),
]

# transposed convolutions, 4x4 stride 2 pad 1: (n, h, w, c_in, c_out)
CONVT = [
    ((1, 65, 66, 256, 512), "data_conv_dma_kernel<false, false>"),
    ((1, 15, 16, 1024, 1024), "data_conv_dma_kernel<128, false, true>"),
    ((8, 32, 32, 256, 128), "data_conv_dma_kernel<128, false, false>"),
    ((2, 40, 40, 72, 256), "data_conv_kernel<Cfg<128, 128, 2, 2>, false, false, false>"),
]

F16_MAX_FINITE = 65504.0
F16_MIN_NORMAL = 2.0 ** -14


def _pixel_pow2(rng, shape, per_element=False):
    """+-2^e per pixel (or per element), e uniform in 0..3, the same for
    every channel of a pixel unless per_element."""
    sz = shape if per_element else shape[:3]
    v = rng.choice([-1.0, 1.0], size=sz) * 2.0 ** rng.integers(0, 4, size=sz)
    if not per_element:
        v = np.broadcast_to(v[..., None], shape)
    return np.ascontiguousarray(v).astype(np.float16)


def _per_channel(n_ch, base):
    """+-base * 2^(j mod 2), the sign flipping every two channels."""
    j = np.arange(n_ch)
    return np.where((j // 2) % 2 == 1, -1.0, 1.0) * (2.0 ** (j % 2)) * base


def _subnormals(rng, shape):
    """Random nonzero multiples of 2^-24 below the smallest normal."""
    m = rng.integers(1, 1024, size=shape) * rng.choice([-1, 1], size=shape)
    return (m * 2.0 ** -24).astype(np.float16)


def _delta(rows, taps_r, taps_s, cols, tap):
    """rows x R x S x cols with a 1 at [i, tap, tap, j] for j = i mod cols."""
    w = np.zeros((rows, taps_r, taps_s, cols), np.float16)
    i = np.arange(rows)
    w[i, tap, tap, i % cols] = 1.0
    return w


def _base_for(o1):
    """Power of two that brings the median magnitude near 0.7 * 65520."""
    med = float(np.median(np.abs(o1[o1 != 0])))
    return 2.0 ** round(np.log2(0.7 * 65520.0 / med))


def _run(op, d, a, b, out_shape, epi, gate):
    ws = workspace(d, fg.OP_CONVT if op == "convT" else op)
    out = empty16(out_shape)
    ga = dev(gate) if gate is not None else None
    if op == FWD:
        fg.conv2d_fwd(d, dev(a), dev(b), out, epi, ga, ws)
    elif op == DX:
        fg.conv2d_bwd_data(d, dev(a), dev(b), out, epi, ga, ws)
    elif op == DW:
        fg.conv2d_bwd_weight(d, dev(a), dev(b), out, ws)
    else:
        fg.conv_transpose2d_fwd(d, dev(a), dev(b), out, epi, ga, ws)
    return host(out)


def _points(op, a, b, shape, idx):
    """Oracle values of the op at flat output indices (a, b as passed to the
    library call)."""
    n, h, w, c, k, r, st, pd = shape
    if op == FWD:
        return oracle.conv2d_fwd_points(a, b, idx, st, pd)
    if op == DX:
        return oracle.conv2d_bwd_data_points(a, b, (n, h, w, c), idx, st, pd)
    if op == DW:
        return oracle.conv2d_bwd_weight_points(a, b, r, r, idx, st, pd)
    return oracle.conv_transpose2d_fwd_points(a, b, idx, st, pd)


def _epilogue(o, epi, gate, idx):
    if epi == fg.EPI_RELU:
        return oracle.relu(o)
    if epi == fg.EPI_GATE:
        return oracle.relu_grad(o, gate.ravel()[idx])
    return o


def _compare(got, o, what):
    with np.errstate(over="ignore"):
        ref = o.astype(np.float16)
    bad = ~((got == ref) | (np.isnan(got) & np.isnan(ref)))
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} differ, e.g. "
                           f"got {got[bad][:4]} expected {ref[bad][:4]} (exact {o[bad][:4]})")
    return ref


def _check(op, shape, kern, recipe):
    n, h, w, c, k, r, st, pd = shape
    if op == "convT":
        d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
        assert fg.kernel_name(d, fg.OP_CONVT) == kern
    else:
        d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
        assert fg.kernel_name(d, op) == kern
    p, q = fg.out_dims(d, op == "convT")
    xs, ys = (n, h, w, c), (n, p, q, k)
    rng = np.random.default_rng(sum(shape) + (7 if recipe == "overflow" else 11))
    # what each op reads (a: data operand, b: the other) and writes
    if op in (FWD, "convT"):
        a_shape, out_shape = xs, ys
        b_shape = (k, r, r, c) if op == FWD else (c, r, r, k)
    elif op == DX:
        a_shape, b_shape, out_shape = ys, (k, r, r, c), xs
    else:
        a_shape, b_shape, out_shape = xs, ys, (k, r, r, c)
    tap = 0 if r == 1 else 1
    epi, gate = fg.EPI_NONE, None
    if recipe == "overflow":
        a = _pixel_pow2(rng, a_shape, per_element=op == DW)
        if op == FWD:
            pat = lambda base: np.broadcast_to(_per_channel(k, base)[:, None, None, None],
                                               b_shape)
        elif op == "convT":
            pat = lambda base: np.broadcast_to(_per_channel(k, base), b_shape)
        elif op == DX:
            pat = lambda base: np.broadcast_to(_per_channel(c, base), b_shape)
            epi = fg.EPI_GATE
            gate = (rng.random(xs) < 0.8).astype(np.float16)
        else:  # kernel gradient: the output gradient depends on k only
            pat = lambda base: np.broadcast_to(_per_channel(k, base), b_shape)
        idx = (np.arange(int(np.prod(out_shape))) if np.prod(out_shape) <= 4096
               else sample_indices(out_shape, 3000, rng))
        o1 = _points(op, a, pat(1.0).astype(np.float16), shape, idx)
        base = _base_for(o1)
        b = np.ascontiguousarray(pat(base)).astype(np.float16)
        assert np.all(np.abs(b[b != 0]) <= F16_MAX_FINITE)
        assert np.array_equal(b.astype(np.float64), pat(base))
        o = o1 * base
    else:
        if op == DW:
            # one nonzero pixel per image, away from the borders
            a = np.zeros(a_shape, np.float16)
            hh, ww = rng.integers(1, h - 1, size=n), rng.integers(1, w - 1, size=n)
            a[np.arange(n), hh, ww, :] = (2.0 ** -12) * (1 + np.arange(c) % 3)
            j = np.arange(k)
            b = np.broadcast_to(np.where(rng.random(k) < 0.5, -1.0, 1.0) * 2.0 ** -8
                                * (1 + j % 2), b_shape).astype(np.float16)
        else:
            a = _subnormals(rng, a_shape)
            if op == FWD:
                b = _delta(k, r, r, c, tap)
                epi = fg.EPI_RELU
            elif op == "convT":
                b = _delta(c, r, r, k, tap)
            else:
                b = _delta(k, r, r, c, tap)
        idx = (np.arange(int(np.prod(out_shape))) if np.prod(out_shape) <= 4096
               else sample_indices(out_shape, 3000, rng))
        o = _points(op, a, b, shape, idx)
    o = _epilogue(o, epi, gate, idx)
    got = _run(op, d, a, b, out_shape, epi, gate).ravel()[idx]
    ref = _compare(got.astype(np.float64), o, f"{kern} {shape} {recipe}")
    if recipe == "overflow":
        assert np.isinf(ref).sum() > 0 and np.isfinite(ref).sum() > 0, kern
        if epi == fg.EPI_NONE:
            assert np.isneginf(ref).any() and np.isposinf(ref).any(), kern
    else:
        sub = (ref != 0) & (np.abs(ref) < F16_MIN_NORMAL)
        assert sub.sum() > 0, kern


@pytest.mark.parametrize("recipe", ["overflow", "subnormal"])
@pytest.mark.parametrize("shape,op,kern", CASES,
                         ids=[f"{['fwd', 'dx', 'dW'][o]}-{k}-{s}" for s, o, k in CASES])
def test_fp16_range_edges(shape, op, kern, recipe):
    _check(op, shape, kern, recipe)


@pytest.mark.parametrize("recipe", ["overflow", "subnormal"])
@pytest.mark.parametrize("shape,kern", CONVT, ids=[f"convT-{k}-{s}" for s, k in CONVT])
def test_fp16_range_edges_convt(shape, kern, recipe):
    n, h, w, ci, co = shape
    _check("convT", (n, h, w, ci, co, 4, 2, 1), kern, recipe)


def test_every_path_is_covered():
    """The cases above reach every kernel name the planner reports for the
    shapes they hold, forward, input gradient, kernel gradient and
    transposed forward alike."""
    names = {k for _, _, k in CASES} | {k for _, k in CONVT}
    for prefix in ("data_conv_dma_kernel<", "data_conv_halo_kernel<",
                   "data_conv_kernel<", "wgrad_dma_kernel<", "wgrad_kernel<", "head_"):
        assert any(nm.startswith(prefix) for nm in names), prefix
    dma = {nm for nm in names if nm.startswith("data_conv_dma_kernel<")}
    assert len(dma) == 8
    halo = {nm for nm in names if nm.startswith("data_conv_halo_kernel<")}
    assert len(halo) == 4
