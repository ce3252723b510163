"""GPU parity of whole workloads: the single conv, the encoder and decoder
blocks, a reduced encoder-decoder step with the gradient path, the full
encoder-decoder step, and that step's gradient path with seeded +inf
injections.

Every op is gated with the single-op rule (rel_L2 <= 5e-3, max_abs <=
2e-2 * RMS, overflow to the same infinity) on its own GPU inputs: the
forward pass of layer i against the oracle applied to the GPU's activation
i, the kernel and input gradients of layer i against the oracle applied to
the GPU's activation i and the GPU's output gradient of layer i. Both sides
then take the same ReLU decisions, and what remains is the rounding of one
op (Section 5.2: three passes per layer). The head gradient, the ReLU
gradient at the top of a block, pack, unscale, unpack and the flags are
bit-exact (Sections 4.2 and 6.2).

Chained values (the oracle propagating its own activations through fp16
storage) are printed as a report, not gated: thirteen layers of last-bit
differences and ReLU decisions on values within an ulp of zero compound,
and no value of the paper pins them.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import chain_report, conv_parity, dev, host, sample_indices
from oracle import chain as OC
from oracle import grad as G
from paper_1909_11150_amd.fcn import Chain

pytestmark = pytest.mark.gpu

S = synth.LOSS_SCALE


def _gate_ops(layers, weights, acts, g, dw, what):
    """Every pass of every layer against the oracle on the GPU's own inputs.
    acts[i] is the GPU's input of layer i (acts[i + 1] its output), g[i + 1]
    the GPU's gradient w.r.t. layer i's pre-activation output, g[i] the input
    gradient layer i wrote, dw[i] its kernel gradient."""
    for i, L in enumerate(layers):
        conv_parity(acts[i + 1], OC.layer_forward(L, acts[i], weights[i]),
                    f"{what} {L.name} fwd")
    for i in reversed(range(len(layers))):
        L = layers[i]
        gate = i > 0 and layers[i - 1].relu
        dx, dwr = OC.layer_backward(L, acts[i], weights[i], g[i + 1], gate)
        conv_parity(dw[i], dwr, f"{what} {L.name} dW")
        conv_parity(g[i], dx, f"{what} {L.name} dx")


def _report_chain(layers, x, weights, acts, dw, dy_top, gate_top):
    """The oracle's own chain (fp16 storage and fp64), printed beside the GPU."""
    o16 = OC.forward(layers, x, weights)
    o64 = OC.forward(layers, x, weights, store_fp16=False)
    dy16 = G.relu_backward(dy_top, o16[-1]) if gate_top else dy_top
    dy64 = np.asarray(dy_top, np.float64)
    if gate_top:
        dy64 = np.where(o64[-1] > 0, dy64, 0.0)
    dws16, _ = OC.backward(layers, o16, weights, dy16)
    dws64, _ = OC.backward(layers, o64, weights, dy64, store_fp16=False)
    for i, L in enumerate(layers):
        chain_report(acts[i + 1], o16[i + 1], o64[i + 1], f"{L.name} act")
        chain_report(dw[i], dws16[i], dws64[i], f"{L.name} dW")


def _run_block(wl):
    ch = Chain(wl.layers, wl.weights, wl.x)
    ch.forward()
    ch.set_output_grad(wl.dy)
    ch.backward()
    acts = [host(a) for a in ch.acts]
    g = [host(t) for t in ch.g]
    dw = [host(t) for t in ch.dw]
    return acts, g, dw


def test_single_conv_workload():
    wl = synth.single_conv()
    L = wl.layers[0]
    acts, g, dw = _run_block(wl)
    np.testing.assert_array_equal(g[1].view(np.uint16), wl.dy.view(np.uint16))
    _gate_ops(wl.layers, wl.weights, acts, g, dw, "single conv")
    assert L.flops == 2 * 2 * 64 * 64 * 16 * 16 * 9


def test_encoder_block_workload():
    """Config 2: both stages' forward, kernel and input gradients, each on
    the GPU's own inputs; the block output's ReLU gradient bit for bit."""
    wl = synth.encoder_block()
    acts, g, dw = _run_block(wl)
    np.testing.assert_array_equal(g[-1].view(np.uint16),
                                  G.relu_backward(wl.dy, acts[-1]).view(np.uint16))
    _gate_ops(wl.layers, wl.weights, acts, g, dw, "encoder block")
    _report_chain(wl.layers, wl.x, wl.weights, acts, dw, wl.dy, True)


def test_decoder_block_workload():
    """Config 3: the transposed conv and the 1x1 conv, all passes, each on
    the GPU's own inputs."""
    wl = synth.decoder_block()
    acts, g, dw = _run_block(wl)
    np.testing.assert_array_equal(g[-1].view(np.uint16), wl.dy.view(np.uint16))
    _gate_ops(wl.layers, wl.weights, acts, g, dw, "decoder block")
    _report_chain(wl.layers, wl.x, wl.weights, acts, dw, wl.dy, False)


def _check_groups(ch, layers, dws_fwd, what):
    """Pack, unscale, unpack and flags of every group, bit for bit against
    the oracle's definitions applied to the given fp16 kernel gradients
    (forward order). Returns the flags."""
    order = list(reversed(range(len(layers))))
    numels = [layers[i].w_numel for i in order]
    srcs = [dws_fwd[i] for i in order]
    plan = G.plan_groups(numels, ch.group_cap_bytes, synth.GROUP_ALIGN_BYTES)
    assert [[order[m] for m in p["members"]] for p in plan] == \
        [g["members"] for g in ch.groups]
    flags = host(ch.flags)
    for gi, p in enumerate(plan):
        ref16 = G.pack(srcs, p)
        np.testing.assert_array_equal(host(ch.gbuf16[gi]).view(np.uint16), ref16,
                                      err_msg=f"{what} G{gi} pack")
        r32, rflag = G.unscale_check(ref16, 1.0 / ch.loss_scale)
        np.testing.assert_array_equal(host(ch.gbuf32[gi]).view(np.uint32),
                                      r32.view(np.uint32), err_msg=f"{what} G{gi} unscale")
        assert flags[gi] == int(rflag), (what, gi, flags)
        for m, v in G.unpack(r32, p, numels).items():
            np.testing.assert_array_equal(host(ch.master[order[m]]).ravel().view(np.uint32),
                                          v.view(np.uint32),
                                          err_msg=f"{what} G{gi} unpack {order[m]}")
    return flags


def test_reduced_network_step_with_gradient_path():
    """Same architecture at 1 x 64 x 64 x 32 with narrower layers, the
    benchmarked step program (three streams), groups capped at 64 KiB so
    that several form, loss scale 2^15: every pass of every layer on its own
    GPU inputs, the head gradient bit for bit on the GPU's output, and the
    gradient path bit for bit on the GPU's kernel gradients."""
    layers = synth.fcn_layers(n=1, h=64, c_in=32, widths=(32, 64, 64, 64),
                              dec=(64, 64, 32, 32))
    x = synth.diffraction_like(1, 64, 32, seed=0)
    w = synth.he_weights(layers, seed=1)
    t = synth.smooth_target(1, 64, seed=4)
    ch = Chain(layers, w, x, loss_scale=S, group_cap_bytes=64 * 1024)
    ch.step(dev(t))
    acts = [host(a) for a in ch.acts]
    g = [host(v) for v in ch.g]
    dw = [host(v) for v in ch.dw]
    np.testing.assert_array_equal(g[-1].view(np.uint16),
                                  G.head_grad(acts[-1], t, S).view(np.uint16))
    _gate_ops(layers, w, acts, g, dw, "reduced step")
    assert len(ch.groups) > 1
    _check_groups(ch, layers, dw, "reduced step")
    _report_chain(layers, x, w, acts, dw, OC.head_grad(OC.forward(layers, x, w)[-1], t, S),
                  False)


# ---- the full network (config 4) and its gradient path (config 5) ----------
@pytest.fixture(scope="module")
def full_step():
    """One run of the benchmarked step program (three streams) on the full
    network; everything it wrote, on the host."""
    wl = synth.fcn()
    ch = Chain(wl.layers, wl.weights, wl.x, loss_scale=S,
               group_cap_bytes=synth.GROUP_CAP_BYTES)
    ch.step(dev(wl.target))
    out = dict(wl=wl, ch=ch,
               acts=[host(a) for a in ch.acts],
               g=[host(v) for v in ch.g],
               dw=[host(v) for v in ch.dw],
               flags=host(ch.flags).copy())
    yield out
    del out["ch"]
    torch.cuda.empty_cache()


def _f64(a):
    return np.asarray(a, dtype=np.float64)


@pytest.mark.parametrize("li", range(13), ids=[L.name for L in synth.fcn_layers()])
def test_full_network_step_each_pass_sampled(full_step, li):
    """Config 4: each of the 39 passes of the benchmarked step, on that
    step's own fp16 tensors, at sampled outputs (all corners included) and
    at every output of the 1x1 head's kernel gradient, whose fp16 value
    overflows to infinity in some channels at loss scale 2^15: there the
    GPU must give the same infinity."""
    wl, acts, g, dw = full_step["wl"], full_step["acts"], full_step["g"], full_step["dw"]
    L = wl.layers[li]
    W = wl.weights[li]
    rng = np.random.default_rng(1000 + li)
    x, dy = _f64(acts[li]), _f64(g[li + 1])
    gate = li > 0 and wl.layers[li - 1].relu
    iy = sample_indices(L.y_shape, 2500, rng)
    ix = sample_indices(L.x_shape, 2500, rng)
    iw = (np.arange(L.w_numel) if L.w_numel <= 4096
          else sample_indices(L.w_shape, 1500, rng))
    if L.kind == "conv":
        fwd = oracle.conv2d_fwd_points(x, W, iy, L.stride, L.pad)
        dxr = oracle.conv2d_bwd_data_points(dy, W, L.x_shape, ix, L.stride, L.pad)
        dwr = oracle.conv2d_bwd_weight_points(x, dy, L.r, L.s, iw, L.stride, L.pad)
    else:
        fwd = oracle.conv_transpose2d_fwd_points(x, W, iy, L.stride, L.pad)
        dxr = oracle.conv2d_fwd_points(dy, W, ix, L.stride, L.pad)
        dwr = oracle.conv2d_bwd_weight_points(dy, x, L.r, L.s, iw, L.stride, L.pad)
    if L.relu:
        fwd = oracle.relu(fwd)
    if gate:
        dxr = np.where(x.ravel()[ix] > 0, dxr, 0.0)
    r = conv_parity(acts[li + 1].ravel()[iy], fwd, f"{L.name} fwd")
    print(f"{L.name} fwd rel_L2 {r[0]:.2e} max/RMS {r[1]:.2e}")
    r = conv_parity(g[li].ravel()[ix], dxr, f"{L.name} dx")
    print(f"{L.name} dx rel_L2 {r[0]:.2e} max/RMS {r[1]:.2e}")
    r = conv_parity(dw[li].ravel()[iw], dwr, f"{L.name} dW")
    print(f"{L.name} dW rel_L2 {r[0]:.2e} max/RMS {r[1]:.2e} infinities {r[2]}")
    if L.name == "F1x1":
        # the head's kernel gradient overflows fp16 at this loss scale
        assert r[2] > 0


def test_full_network_head_gradient_and_groups(full_step):
    """Config 4/5 without injection: the head gradient bit for bit on the
    step's own output; every group buffer, fp32 master gradient and flag bit
    for bit on the step's own kernel gradients."""
    wl, ch = full_step["wl"], full_step["ch"]
    acts, g = full_step["acts"], full_step["g"]
    np.testing.assert_array_equal(g[-1].view(np.uint16),
                                  G.head_grad(acts[-1], wl.target, S).view(np.uint16))
    assert len(ch.groups) == 9
    flags = _check_groups(ch, wl.layers, full_step["dw"], "config 4")
    np.testing.assert_array_equal(flags, full_step["flags"])


def test_config5_injection_into_the_step_gradients(full_step):
    """Config 5: 99 seeded +inf values (1 in 10^6 of the 99,483,904
    gradient elements, seed 7, flat positions over the tensors in backward
    completion order) written into the step's own fp16 kernel gradients
    after the backward pass; then each group's pack, unscale and unpack.
    Group buffers, fp32 master gradients and flags bit for bit against the
    oracle; the flagged groups are exactly those holding an injection or a
    kernel gradient that overflowed by itself."""
    wl, ch = full_step["wl"], full_step["ch"]
    layers = wl.layers
    order = list(reversed(range(len(layers))))
    numels = [layers[i].w_numel for i in order]
    bounds = np.cumsum([0] + numels)
    inj = synth.injection_indices(int(bounds[-1]))
    assert inj.size == 99
    natural = {i for i in range(len(layers))
               if not np.all(np.isfinite(full_step["dw"][i]))}
    hit = set()
    for j, i in enumerate(order):
        sel = inj[(inj >= bounds[j]) & (inj < bounds[j + 1])] - bounds[j]
        if sel.size:
            ch.dw[i].view(-1)[torch.from_numpy(sel).to(ch.dw[i].device)] = float("inf")
            hit.add(i)
    ch.flags.zero_()
    for gi in range(len(ch.groups)):
        ch.run_group(gi)
    dw = [host(v) for v in ch.dw]
    for i in hit:
        assert np.isposinf(dw[i]).sum() >= 1
    flags = _check_groups(ch, layers, dw, "config 5")
    expect = [int(any(m in hit or m in natural for m in g["members"]))
              for g in ch.groups]
    np.testing.assert_array_equal(flags, expect)
    assert sum(expect) >= 1


def test_full_network_step_is_deterministic(full_step):
    """A second run of the step program gives the bits of the first."""
    wl, ch = full_step["wl"], full_step["ch"]
    # the injection test may have changed dW and the group buffers: a new
    # step recomputes everything from the activations up
    ch.step(dev(wl.target))
    for a, b in zip(full_step["acts"][1:], ch.acts[1:]):
        assert np.array_equal(a.view(np.uint16), host(b).view(np.uint16))
    for a, b in zip(full_step["dw"], ch.dw):
        assert np.array_equal(a.view(np.uint16), host(b).view(np.uint16))
    np.testing.assert_array_equal(full_step["flags"], host(ch.flags))
