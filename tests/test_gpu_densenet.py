"""GPU parity of the FC-DenseNet variant (Section 6.2): the reduced network's
whole step against the oracle network, every full-size layer shape on
sampled outputs, and the full-size step's determinism.

Reduced step: the oracle runs the same network from the same inputs with
fp16 storage at the same points (O16) and entirely in fp64 (O64). Per-op
differences propagate through the chain, so chained outputs are held to
rel_L2(GPU, O16) <= max(5e-3, 2 rel_L2(O16, O64)), the rule of the chain
tests. The backward pass is checked on the GPU's own forward tensors, so
that a ReLU decision flipped by a last-bit difference of the forward pass
does not enter the gradients' comparison; the Huber head gradient of the
GPU's own output is compared bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import chain_parity, conv_parity, dev, host, sample_indices
from oracle import dense as D
from oracle import dense_net as DN
from paper_1909_11150_amd import fcn
from paper_1909_11150_amd.densenet import DenseNet
import paper_1909_11150_amd as fg

pytestmark = pytest.mark.gpu

S_RED = 2.0 ** 10
DELTA = 10.0


def _reduced():
    layers = synth.densenet_layers(n=1, h=32, c_in=32, c0=32, growth=32, levels=2,
                                   per_block=2)
    x = synth.diffraction_like(1, 32, 32, seed=0)
    w = synth.he_weights(layers, seed=1)
    t = synth.smooth_target(1, 32, seed=4) * np.float32(3.0)
    return layers, x, w, t


def _gpu_forward_state(net):
    """The GPU's stored forward tensors, keyed as the oracle network's: each
    layer's input and output are views of the network's level buffers. The
    last concatenation of the bottleneck and up blocks, which nothing reads
    and the GPU does not keep, is rebuilt on the host from the block's
    tensors (the oracle's backward pass takes only its shape)."""
    view = lambda s: host(net._view(s))
    fw = {name: host(a) for name, a in net.act.items()}
    fw["y"] = fw["F1x1"]
    lv, per = net.levels, net.per
    for d in range(1, lv + 1):
        fw[f"P{d}"] = host(net.P[d])
        fw[f"in:TU{d}"] = host(net.NF["B" if d == lv else f"U{d + 1}"])
        fw[f"skip{d}"] = fw[f"Z:D{d}:{per}"] = view(net.inp[f"TD{d}"])
    for blk in net._blocks():
        for l in range(1, per + 1):
            fw[f"Z:{blk}:{l - 1}"] = view(net.inp[f"{blk}.{l}"])
        if not blk.startswith("D"):
            fw[f"Z:{blk}:{per}"] = np.concatenate([fw[f"Z:{blk}:{per - 1}"],
                                                   fw[f"{blk}.{per}"]], axis=-1)
    fw["in:F1x1"] = host(net.NF["U1"])
    return fw


def test_reduced_densenet_step():
    """Forward: chained activations against the oracle network. Backward:
    the oracle's backward pass run on the GPU's own forward tensors and head
    gradient (so both sides take the same ReLU decisions), kernel and input
    gradients held to the chain rule against that pass in fp16 storage and
    in fp64."""
    layers, x, w, t = _reduced()
    net = DenseNet(layers, w, x, loss_scale=S_RED, delta=DELTA)
    net.step(dev(t))
    torch.cuda.synchronize()
    y = host(net.act["F1x1"])
    # head gradient on the GPU's own output: bit for bit
    g_ref = D.huber_head_grad(y, t, S_RED / y.size, DELTA)
    g_gpu = host(net.g_out)
    np.testing.assert_array_equal(g_gpu.view(np.uint16), g_ref.view(np.uint16))
    f16 = DN.forward(layers, x, w)
    f64 = DN.forward(layers, x, w, store_fp16=False)
    for L in layers:
        key = "y" if L.name == "F1x1" else L.name
        chain_parity(host(net.act[L.name]), f16[key], f64[key], None, f"{L.name} act")
    for d in (1, 2):
        chain_parity(host(net.P[d]), f16[f"P{d}"], f64[f"P{d}"], None, f"P{d}")
    fw = _gpu_forward_state(net)
    dW16, dX16 = DN.backward(layers, fw, x, w, g_gpu)
    dW64, dX64 = DN.backward(layers, fw, x, w, g_gpu, store_fp16=False)
    for L in layers:
        chain_parity(host(net.dw[L.name]), dW16[L.name], dW64[L.name], None, f"{L.name} dW")
    chain_parity(host(net.dX), dX16, dX64, None, "dX")


def test_reduced_densenet_program_is_deterministic():
    layers, x, w, t = _reduced()
    net = DenseNet(layers, w, x, loss_scale=S_RED, delta=DELTA)
    td = dev(t)
    outs = []
    for _ in range(2):
        net.step(td)
        outs.append({k: host(v).view(np.uint16).copy() for k, v in net.dw.items()})
    for k in outs[0]:
        assert np.array_equal(outs[0][k], outs[1][k]), k


def test_streams_match_one_stream():
    """Kernel gradients on a second stream, and concatenation copies on a
    third, give the bits of the one-stream order, over two steps."""
    layers, x, w, t = _reduced()
    td = dev(t)
    out = []
    for streams in (1, 2, 3):
        net = DenseNet(layers, w, x, loss_scale=S_RED, delta=DELTA)
        prog = net.program(td, streams=streams)
        assert len(prog.streams) == streams
        for _ in range(2):
            prog.run()
        prog.join()
        torch.cuda.synchronize()
        out.append({k: host(v).view(np.uint16).copy() for k, v in net.dw.items()})
        out[-1]["dX"] = host(net.dX).view(np.uint16).copy()
    for o in out[1:]:
        for k in out[0]:
            assert np.array_equal(out[0][k], o[k]), k


def _unique_layers():
    seen, out = set(), []
    for L in synth.densenet_layers():
        key = (L.kind, L.x_shape, L.y_shape, L.r, L.stride)
        if key not in seen:
            seen.add(key)
            out.append(L)
    return out


LAYERS = _unique_layers()


@pytest.mark.parametrize("L", LAYERS, ids=[L.name for L in LAYERS])
def test_full_size_dense_layer_sampled(L):
    """Each full-size layer shape of the dense network: forward (+ ReLU),
    input gradient and kernel gradient on sampled outputs."""
    rng = np.random.default_rng(LAYERS.index(L) + 300)
    x = np.maximum(synth.normal(rng, L.x_shape), np.float16(0))
    w = synth.normal(rng, L.w_shape, synth.he_std(L))
    dy = synth.normal(rng, L.y_shape, 1.0)
    dx_, w_, dy_ = dev(x), dev(w), dev(dy)
    y = torch.empty(L.y_shape, dtype=torch.float16, device="cuda")
    dx = torch.empty(L.x_shape, dtype=torch.float16, device="cuda")
    dw = torch.empty(L.w_shape, dtype=torch.float16, device="cuda")
    ws = torch.empty(max(16, fcn.chain_workspace_bytes([L])), dtype=torch.uint8,
                     device="cuda")
    epi = fg.EPI_RELU if L.relu else fg.EPI_NONE
    srng = np.random.default_rng(8)
    iy = sample_indices(L.y_shape, 2000, srng)
    ix = sample_indices(L.x_shape, 2000, srng)
    iw = sample_indices(L.w_shape, 1000, srng)
    if L.kind == "conv":
        d = fcn.fwd_desc(L)
        fg.conv2d_fwd(d, dx_, w_, y, epi, None, ws)
        fg.conv2d_bwd_data(d, dy_, w_, dx, fg.EPI_NONE, None, ws)
        fg.conv2d_bwd_weight(d, dx_, dy_, dw, ws)
        ref = oracle.conv2d_fwd_points(x, w, iy, L.stride, L.pad)
        rx = oracle.conv2d_bwd_data_points(dy, w, x.shape, ix, L.stride, L.pad)
        rw = oracle.conv2d_bwd_weight_points(x, dy, L.r, L.s, iw, L.stride, L.pad)
    else:
        fg.conv_transpose2d_fwd(fcn.fwd_desc(L), dx_, w_, y, epi, None, ws)
        dd = fcn.convt_dx_desc(L)
        fg.conv2d_fwd(dd, dy_, w_, dx, fg.EPI_NONE, None, ws)
        fg.conv2d_bwd_weight(dd, dy_, dx_, dw, ws)
        ref = oracle.conv_transpose2d_fwd_points(x, w, iy, L.stride, L.pad)
        rx = oracle.conv2d_fwd_points(dy, w, ix, L.stride, L.pad)
        rw = oracle.conv2d_bwd_weight_points(dy, x, L.r, L.s, iw, L.stride, L.pad)
    if L.relu:
        ref = oracle.relu(ref)
    conv_parity(host(y).ravel()[iy], ref, f"{L.name} fwd")
    conv_parity(host(dx).ravel()[ix], rx, f"{L.name} dx")
    conv_parity(host(dw).ravel()[iw], rw, f"{L.name} dW")


def test_full_densenet_step_is_deterministic_and_finite():
    wl = synth.densenet()
    net = DenseNet(wl.layers, wl.weights, wl.x, loss_scale=2.0 ** 12, delta=DELTA)
    td = dev(wl.target)
    outs = []
    for _ in range(2):
        net.step(td)
        torch.cuda.synchronize()
        outs.append({k: host(v).view(np.uint16).copy() for k, v in net.dw.items()})
    for k in outs[0]:
        assert np.array_equal(outs[0][k], outs[1][k]), k
    for name, a in net.act.items():
        assert np.all(np.isfinite(host(a).astype(np.float32))), name
    assert np.all(np.isfinite(host(net.dX).astype(np.float32)))


def test_densenet_gradient_groups():
    """The dense step's gradient path: kernel gradients packed into groups
    in completion order (bits and zero padding), unscaled with the
    non-finite check and unpacked into fp32 master gradients, against the
    oracle's definitions applied to the step's own kernel gradients."""
    from oracle import grad as OG
    layers, x, w, t = _reduced()
    net = DenseNet(layers, w, x, loss_scale=S_RED, delta=DELTA, group_cap_bytes=48 * 1024,
                   group_align_bytes=256)
    assert len(net.groups) >= 3
    order = net.dw_order()
    assert [m for g in net.groups for m in g["members"]] == order
    plan = OG.plan_groups([net.dw[m].numel() for m in order], 48 * 1024, 256)
    assert [g["numel"] for g in plan] == [g["numel"] for g in net.groups]
    net.step(dev(t))
    torch.cuda.synchronize()
    inv = np.float32(1.0 / S_RED)
    flags = host(net.flags)
    for gi, g in enumerate(net.groups):
        g16 = host(net.gbuf16[gi]).view(np.uint16)
        want = np.zeros(g["numel"], np.uint16)
        src = {}
        for m, off in zip(g["members"], g["offsets"]):
            src[m] = host(net.dw[m]).ravel().view(np.uint16)
            want[off:off + src[m].size] = src[m]
        np.testing.assert_array_equal(g16, want)
        np.testing.assert_array_equal(host(net.gbuf32[gi]).view(np.uint32),
                                      OG.unscale(want, inv).view(np.uint32))
        assert int(flags[gi]) == int(OG.found_nonfinite(want))
        for m in g["members"]:
            np.testing.assert_array_equal(host(net.master[m]).ravel().view(np.uint32),
                                          OG.unscale(src[m], inv).view(np.uint32))
