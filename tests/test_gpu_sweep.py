"""Seeded random-shape sweep of the convolution passes against the fp64
oracle (Section 5.2: forward, input-gradient and kernel-gradient passes of
every layer).

The other GPU tests pin each kernel path on chosen shapes. This one draws
shapes the library accepts at random (a fixed seed, so the cases are the same
on every run): kernel sizes 1..4 per axis with r*s <= 16 (1x3, 2x4 and
other non-square ones too), strides 1..3 (input gradients 1..2), any padding
below the kernel size, channels any multiple of 8, images from 1x1 up, so
that the planner's choices meet shapes nobody picked: empty output phases of
strided input gradients, images smaller than the kernel, single-tile and
ragged tiles, split and unsplit reductions. Small cases are compared in
full; large ones (on the LDS-DMA, halo and split kernels) on sampled outputs
plus all corners; each call is made twice and must give the same bits. The parity rule is the one every convolution test uses
(rel_L2 <= 5e-3 and max_abs <= 2e-2 * RMS against the fp64 oracle on the
same fp16 inputs).
"""
import zlib

import numpy as np
import pytest

import oracle
import paper_1909_11150_amd as fg
import synth
from gpu_util import conv_parity, dev, empty16, host, sample_indices, workspace

pytestmark = pytest.mark.gpu

FWD, DX, DW, CT = fg.OP_FWD, fg.OP_BWD_DATA, fg.OP_BWD_WEIGHT, fg.OP_CONVT
EPI = {"none": fg.EPI_NONE, "relu": fg.EPI_RELU, "gate": fg.EPI_GATE}
CHANNELS_SMALL = (8, 16, 24, 40, 64, 72, 96, 128, 136)
CHANNELS_LARGE = (256, 512, 264, 384)
FULL_FLOPS = 4e8      # above this, sampled outputs only
SAMPLES = 1500


def _out(h, pad, r, stride):
    return (h + 2 * pad - r) // stride + 1


def draw_cases(seed=20191125, n_small=90, n_large=30, n_layer=30):
    """(op, (n, h, w, c, k, r, s, stride, pad)) cases, all of which the
    library accepts: c, k multiples of 8, r*s <= 16, output at least 1x1,
    input-gradient strides at most 2. Three groups: small shapes of any kind,
    large ones of any kind, and layer-like ones (square 3x3 or 4x4 kernels,
    padding 1, widths 32, 64 or 128 and 256 or 512 channels, the shapes that
    take the 256 x 256 and halo kernels) with random heights and batch."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n_small + n_large + n_layer:
        group = 0 if len(cases) < n_small else 1 if len(cases) < n_small + n_large else 2
        op = (FWD, DX, DW)[len(cases) % 3]
        r, s = (int(v) for v in rng.integers(1, 5, size=2))
        if r * s > 16:
            continue
        stride = int(rng.integers(1, 3 if op == DX else 4))
        pad = int(rng.integers(0, min(r, s)))
        if group == 2:
            r = s = int(rng.choice((3, 3, 4)))
            stride, pad = int(rng.choice((1, 1, 2))), 1
            c, k = (int(rng.choice((256, 512))) for _ in range(2))
            n = int(rng.integers(1, 5))
            w = int(rng.choice((32, 64, 128))) * stride
            h = int(rng.integers(8, 80)) * stride
        elif group == 1:
            c, k = (int(rng.choice(CHANNELS_LARGE)) for _ in range(2))
            n = int(rng.integers(1, 4))
            h, w = (int(v) for v in rng.integers(24, 140, size=2))
        else:
            c, k = (int(rng.choice(CHANNELS_SMALL)) for _ in range(2))
            n = int(rng.integers(1, 4))
            h, w = (int(v) for v in rng.integers(1, 34, size=2))
        if _out(h, pad, r, stride) < 1 or _out(w, pad, s, stride) < 1:
            continue
        cases.append((op, (n, h, w, c, k, r, s, stride, pad)))
    return cases


def draw_convt(seed=20191126, count=18):
    """Transposed convolutions (4x4, stride 2, padding 1, the decoder's):
    (n, h, w, c_in, c_out), half of them small, half large."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        if i < count // 2:
            c, k = (int(rng.choice(CHANNELS_SMALL)) for _ in range(2))
            n = int(rng.integers(1, 4))
            h, w = (int(v) for v in rng.integers(1, 24, size=2))
        else:
            c, k = (int(rng.choice(CHANNELS_LARGE + (1024,))) for _ in range(2))
            n = int(rng.integers(1, 4))
            h, w = (int(v) for v in rng.integers(8, 70, size=2))
        out.append((n, h, w, c, k))
    return out


def epilogue_of(name):
    """The epilogue a case runs: drawn from its name (forward: none, ReLU or
    gate; input gradient: none or gate; kernel gradient: none)."""
    v = zlib.crc32(("epi" + name).encode())
    if name.startswith(("fwd", "convT")):
        return ("none", "relu", "gate")[v % 3]
    if name.startswith("dx"):
        return ("none", "gate")[v % 2]
    return "none"


CASES = draw_cases()
CONVT = draw_convt()


def _name(case):
    op, (n, h, w, c, k, r, s, st, pd) = case
    return f"{['fwd', 'dx', 'dW'][op]}-n{n}-{h}x{w}-c{c}-k{k}-{r}x{s}-s{st}-p{pd}"


def check_coverage():
    """The draw reaches the register-staged, LDS-DMA, halo and split kernels
    and the strided, non-square and empty-phase corners (run by the CPU
    tests: it needs the planner only)."""
    names = set()
    for op, (n, h, w, c, k, r, s, st, pd) in CASES:
        names.add(fg.kernel_name(fg.ConvDesc.make(n, h, w, c, k, r, s, st, pd), op))
    ct = {fg.kernel_name(fg.ConvDesc.make(n, h, w, c, k, 4, 4, 2, 1), CT)
          for n, h, w, c, k in CONVT}
    assert any(nm.startswith("data_conv_dma_kernel<false") for nm in ct), ct
    assert any(nm.startswith("data_conv_kernel<") for nm in ct), ct
    epis = {epilogue_of(_name(c)) for c in CASES}
    assert epis == {"none", "relu", "gate"}, epis
    joined = " ".join(sorted(names))
    for fam in ("data_conv_kernel<", "data_conv_dma_kernel<true", "data_conv_dma_kernel<false",
                "data_conv_dma_kernel<128", "data_conv_halo_kernel<", "wgrad_kernel<",
                "wgrad_dma_kernel<true>"):
        assert fam in joined, (fam, sorted(names))
    assert any(r != s for _, (_, _, _, _, _, r, s, _, _) in CASES)
    assert any(st == 2 and op == DX for op, (*_, st, _) in CASES)
    # an input gradient with an output phase that no tap reaches
    assert any(op == DX and st == 2 and (r == 1 or s == 1)
               for op, (_, _, _, _, _, r, s, st, _) in CASES)


@pytest.mark.parametrize("case", CASES, ids=[_name(c) for c in CASES])
def test_random_shape_parity(case):
    op, (n, h, w, c, k, r, s, st, pd) = case
    d = fg.ConvDesc.make(n, h, w, c, k, r, s, st, pd)
    kern = fg.kernel_name(d, op)
    print(f"{_name(case)}: {kern}", flush=True)
    p, q = _out(h, pd, r, st), _out(w, pd, s, st)
    rng = np.random.default_rng(zlib.crc32(_name(case).encode()))
    x = synth.uniform(rng, (n, h, w, c))
    W = synth.normal(rng, (k, r, s, c), np.sqrt(2.0 / (r * s * c)))
    dy = synth.uniform(rng, (n, p, q, k))
    flops = 2.0 * n * p * q * k * c * r * s
    full = flops <= FULL_FLOPS
    ws = workspace(d, op)
    epi = epilogue_of(_name(case))
    if op == FWD:
        out = empty16((n, p, q, k))
        gate = synth.uniform(rng, out.shape) if epi == "gate" else None
        call = lambda o: fg.conv2d_fwd(d, dev(x), dev(W), o, EPI[epi],
                                       dev(gate) if gate is not None else None, ws)
        call(out)
        if full:
            ref = oracle.conv2d_fwd(x, W, st, pd)
        else:
            idx = sample_indices(out.shape, SAMPLES, rng)
            ref = oracle.conv2d_fwd_points(x, W, idx, st, pd)
    elif op == DX:
        out = empty16(x.shape)
        gate = synth.uniform(rng, out.shape) if epi == "gate" else None
        call = lambda o: fg.conv2d_bwd_data(d, dev(dy), dev(W), o, EPI[epi],
                                            dev(gate) if gate is not None else None, ws)
        call(out)
        if full:
            ref = oracle.conv2d_bwd_data(dy, W, x.shape, st, pd)
        else:
            idx = sample_indices(out.shape, SAMPLES, rng)
            ref = oracle.conv2d_bwd_data_points(dy, W, x.shape, idx, st, pd)
    else:
        out = empty16(W.shape)
        call = lambda o: fg.conv2d_bwd_weight(d, dev(x), dev(dy), o, ws)
        call(out)
        if full:
            ref = oracle.conv2d_bwd_weight(x, dy, r, s, st, pd)
        else:
            idx = sample_indices(out.shape, SAMPLES, rng)
            ref = oracle.conv2d_bwd_weight_points(x, dy, r, s, idx, st, pd)
    got = host(out)
    # a second call, into a fresh buffer, gives the same bits (every sum in
    # a fixed order, split reductions included)
    again = empty16(out.shape)
    call(again)
    assert np.array_equal(host(again).view(np.uint16), got.view(np.uint16)), _name(case)
    if not full:
        got = got.ravel()[idx]
    if epi != "none":
        g = None if gate is None else (gate if full else gate.ravel()[idx])
        ref = _epilogue(ref, epi, g)
    conv_parity(got, ref, f"{_name(case)} {epi} ({kern})")


def _epilogue(acc, epi, gate):
    """The oracle's epilogue for the case: ReLU, or the ReLU-gradient gate."""
    return oracle.relu(acc) if epi == "relu" else oracle.relu_grad(acc, gate)


def _convt_name(t):
    n, h, w, c, k = t
    return f"convT-n{n}-{h}x{w}-c{c}-k{k}"


@pytest.mark.parametrize("t", CONVT, ids=[_convt_name(t) for t in CONVT])
def test_random_shape_convt_parity(t):
    n, h, w, c, k = t
    d = fg.ConvDesc.make(n, h, w, c, k, 4, 4, 2, 1)
    kern = fg.kernel_name(d, CT)
    name = _convt_name(t)
    print(f"{name}: {kern}", flush=True)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    x = synth.uniform(rng, (n, h, w, c))
    Wt = synth.normal(rng, (c, 4, 4, k), np.sqrt(2.0 / (4 * c)))
    out = empty16((n, 2 * h, 2 * w, k))
    epi = epilogue_of(name)
    gate = synth.uniform(rng, out.shape) if epi == "gate" else None
    fg.conv_transpose2d_fwd(d, dev(x), dev(Wt), out, EPI[epi],
                            dev(gate) if gate is not None else None, workspace(d, CT))
    full = 2.0 * n * h * w * c * k * 16 <= FULL_FLOPS
    if full:
        ref, got, g = oracle.conv_transpose2d_fwd(x, Wt, 2, 1), host(out), gate
    else:
        idx = sample_indices(out.shape, SAMPLES, rng)
        ref = oracle.conv_transpose2d_fwd_points(x, Wt, idx, 2, 1)
        got = host(out).ravel()[idx]
        g = None if gate is None else gate.ravel()[idx]
    if epi != "none":
        ref = _epilogue(ref, epi, g)
    conv_parity(got, ref, f"{name} {epi} ({kern})")


SLICED = CASES[::4]


@pytest.mark.parametrize("case", SLICED, ids=[_name(c) for c in SLICED])
def test_random_shape_channel_slices(case):
    """The same pass with its output in a channel slice of a wider buffer
    (pixel stride = channels + 8a, slice at channel 8b, b <= a), and the
    forward pass and kernel gradient reading x from such a slice (the
    layouts a dense block's concatenation uses): the slice holds the dense
    call's bits and every other channel keeps its own."""
    op, (n, h, w, c, k, r, s, st, pd) = case
    name = _name(case)
    rng = np.random.default_rng(zlib.crc32(("slice" + name).encode()))
    p, q = _out(h, pd, r, st), _out(w, pd, s, st)
    a_in, a_out = (int(v) for v in rng.integers(0, 4, size=2))
    b_in, b_out = int(rng.integers(0, a_in + 1)), int(rng.integers(0, a_out + 1))
    ld_in, ld_out = c + 8 * a_in, (k if op != DX else c) + 8 * a_out
    dense = fg.ConvDesc.make(n, h, w, c, k, r, s, st, pd)
    # the output's pixel stride: y_ld for the forward pass, x_ld for the
    # input gradient; x read from a slice by the forward pass and kernel gradient
    if op == FWD:
        sliced = fg.ConvDesc.make(n, h, w, c, k, r, s, st, pd, x_ld=ld_in, y_ld=ld_out)
    elif op == DX:
        sliced = fg.ConvDesc.make(n, h, w, c, k, r, s, st, pd, x_ld=ld_out)
    else:
        sliced = fg.ConvDesc.make(n, h, w, c, k, r, s, st, pd, x_ld=ld_in)
    kern = fg.kernel_name(dense, op)
    assert fg.kernel_name(sliced, op) == kern
    print(f"{name}: {kern}, in ld {ld_in} at {8 * b_in}, out ld {ld_out} at {8 * b_out}",
          flush=True)
    x = synth.uniform(rng, (n, h, w, c))
    W = synth.normal(rng, (k, r, s, c), np.sqrt(2.0 / (r * s * c)))
    dy = synth.uniform(rng, (n, p, q, k))
    # the wide input: x in channels [8 b_in, 8 b_in + c), other channels random
    wide_in = synth.uniform(rng, (n, h, w, ld_in))
    wide_in[..., 8 * b_in:8 * b_in + c] = x
    x_wide = dev(wide_in)
    x_slice = x_wide.view(-1)[8 * b_in:]  # the slice's first element
    if op == DW:
        ref, got = empty16(W.shape), empty16(W.shape)
        fg.conv2d_bwd_weight(dense, dev(x), dev(dy), ref, workspace(dense, op))
        fg.conv2d_bwd_weight(sliced, x_slice, dev(dy), got, workspace(sliced, op))
        assert np.array_equal(host(got).view(np.uint16), host(ref).view(np.uint16)), name
        return
    oshape = (n, p, q, k) if op == FWD else (n, h, w, c)
    och = oshape[3]
    fill = synth.uniform(rng, oshape[:3] + (ld_out,))
    out_wide = dev(fill)
    out_slice = out_wide.view(-1)[8 * b_out:]
    ref = empty16(oshape)
    if op == FWD:
        fg.conv2d_fwd(dense, dev(x), dev(W), ref, fg.EPI_RELU, None, workspace(dense, op))
        fg.conv2d_fwd(sliced, x_slice, dev(W), out_slice, fg.EPI_RELU, None,
                      workspace(sliced, op))
    else:
        fg.conv2d_bwd_data(dense, dev(dy), dev(W), ref, fg.EPI_NONE, None,
                           workspace(dense, op))
        fg.conv2d_bwd_data(sliced, dev(dy), dev(W), out_slice, fg.EPI_NONE, None,
                           workspace(sliced, op))
    got = host(out_wide).view(np.uint16)
    inside = np.zeros(ld_out, bool)
    inside[8 * b_out:8 * b_out + och] = True
    assert np.array_equal(got[..., inside], host(ref).view(np.uint16)), name
    assert np.array_equal(got[..., ~inside], fill.view(np.uint16)[..., ~inside]), name


def draw_heads(seed=20191127, count=12):
    """The K = 1 head (1x1, stride 1, no padding; its own bandwidth kernels):
    (n, h, w, c) with c any multiple of 8 up to 2048."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        t = (int(rng.integers(1, 5)), int(rng.integers(1, 300)), int(rng.integers(1, 300)),
             8 * int(rng.integers(1, 257)))
        if np.prod(t) <= 1 << 25:  # host memory of the fp64 oracle
            out.append(t)
    return out


HEADS = draw_heads()


@pytest.mark.parametrize("t", HEADS, ids=[f"head-n{n}-{h}x{w}-c{c}" for n, h, w, c in HEADS])
def test_random_head_parity(t):
    """Forward (ReLU'd activations as the head's input), input gradient
    gated by the activations (one product per output: the oracle rounded
    once to fp16, exactly) and kernel gradient (a sum over every position)."""
    n, h, w, c = t
    rng = np.random.default_rng(zlib.crc32(f"head{t}".encode()))
    x = np.maximum(synth.uniform(rng, (n, h, w, c)), np.float16(0))
    W = synth.normal(rng, (1, 1, 1, c), np.sqrt(2.0 / c))
    dy = synth.uniform(rng, (n, h, w, 1))
    d = fg.ConvDesc.make(n, h, w, c, 1, 1, 1, 1, 0)
    print(f"head {t}: {fg.kernel_name(d, FWD)}, {fg.kernel_name(d, DX)}, "
          f"{fg.kernel_name(d, DW)}", flush=True)
    y = empty16((n, h, w, 1))
    fg.conv2d_fwd(d, dev(x), dev(W), y, fg.EPI_NONE, None, workspace(d, FWD))
    conv_parity(host(y), oracle.conv2d_fwd(x, W, 1, 0), f"head fwd {t}")
    dx = empty16(x.shape)
    fg.conv2d_bwd_data(d, dev(dy), dev(W), dx, fg.EPI_GATE, dev(x), workspace(d, DX))
    ref = oracle.conv2d_bwd_data(dy, W, x.shape, 1, 0, epi="gate", gate=x)
    np.testing.assert_array_equal(host(dx), ref.astype(np.float16))  # +0 == -0
    dw = empty16(W.shape)
    fg.conv2d_bwd_weight(d, dev(x), dev(dy), dw, workspace(d, DW))
    conv_parity(host(dw), oracle.conv2d_bwd_weight(x, dy, 1, 1, 1, 0), f"head dW {t}")
