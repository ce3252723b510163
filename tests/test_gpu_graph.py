"""The library's calls captured in a HIP graph: every replay reproduces the
eager results bit for bit, with eager work and synchronisations between the
replays (a captured memset node, or any state a call leaves behind for the
next, would show here). Two cases: a small block's forward and backward pass
on one stream, and the reduced encoder-decoder's three-stream step program
with its gradient groups."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import dev, host
from paper_1909_11150_amd.fcn import Chain

pytestmark = pytest.mark.gpu


def _bits(ts):
    torch.cuda.synchronize()
    return [host(t).view(np.uint8).copy() for t in ts]


def _same(a, b):
    return all(np.array_equal(x, y) for x, y in zip(a, b))


def test_block_pass_replays_bit_exact():
    wl = synth.encoder_block()
    ch = Chain(wl.layers, wl.weights, wl.x)
    ch.set_output_grad(wl.dy)
    outs = ch.acts[1:] + ch.g[:-1] + ch.dw

    def step():
        ch.forward()
        ch.backward()
    step()
    ref = _bits(outs)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for _ in range(3):
        for t in outs:
            t.zero_()
        g.replay()
        assert _same(ref, _bits(outs))
        step()  # eager work between replays
        assert _same(ref, _bits(outs))


def test_three_stream_step_program_replays_bit_exact():
    layers = synth.fcn_layers(n=1, h=64, c_in=32, widths=(32, 64, 64, 64),
                              dec=(64, 64, 32, 32))
    x = synth.diffraction_like(1, 64, 32, seed=0)
    w = synth.he_weights(layers, seed=1)
    t = dev(synth.smooth_target(1, 64, seed=4))
    cap = torch.cuda.Stream()
    ch = Chain(layers, w, x, loss_scale=synth.LOSS_SCALE, group_cap_bytes=64 * 1024,
               stream=cap.cuda_stream)
    prog = ch.program(t, streams=3)
    outs = ch.acts[1:] + ch.master + ch.gbuf16 + [ch.flags]
    with torch.cuda.stream(cap):
        prog.run()
        prog.join()
    ref = _bits(outs)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        prog.run()
        prog.join()
    for _ in range(3):
        for o in outs:
            o.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(cap):
            g.replay()
        assert _same(ref, _bits(outs))
        with torch.cuda.stream(cap):  # eager work between replays
            prog.run()
            prog.join()
        assert _same(ref, _bits(outs))
