"""GPU checks of the step program's options and of the library's measurement
and flag helpers: kernel gradients released in batches give the bits of the
per-layer release; the main-kernel events of fg_profile_next_launch bracket
the main kernel only (inside the call, before a split reduction); the flag
clear zeroes exactly its range."""
import numpy as np
import pytest
import torch

import paper_1909_11150_amd as fg
import synth
from gpu_util import dev, empty16, host, workspace
from paper_1909_11150_amd.fcn import Chain

pytestmark = pytest.mark.gpu


def _reduced_chain():
    layers = synth.fcn_layers(n=1, h=64, c_in=32, widths=(32, 64, 64, 64),
                              dec=(64, 64, 32, 32))
    x = synth.diffraction_like(1, 64, 32, seed=0)
    w = synth.he_weights(layers, seed=1)
    t = synth.smooth_target(1, 64, seed=4)
    ch = Chain(layers, w, x, loss_scale=synth.LOSS_SCALE, group_cap_bytes=64 * 1024)
    return ch, dev(t)


def _snap(ch):
    torch.cuda.synchronize()
    return ([host(a).view(np.uint16).copy() for a in ch.acts[1:]] +
            [host(m).view(np.uint32).copy() for m in ch.master] +
            [host(g).view(np.uint16).copy() for g in ch.gbuf16] + [host(ch.flags).copy()])


@pytest.mark.parametrize("sync_every", [2, 3, 13])
def test_batched_kernel_gradient_release_gives_the_same_bits(sync_every):
    ch, t = _reduced_chain()
    ref_prog = ch.program(t, streams=1)
    ref_prog.run()
    ref_prog.join()
    ref = _snap(ch)
    for a in ch.master:
        a.zero_()
    prog = ch.program(t, streams=3, sync_every=sync_every)
    for _ in range(2):
        prog.run()
    prog.join()
    got = _snap(ch)
    assert all(np.array_equal(a, b) for a, b in zip(ref, got))
    # every kernel gradient waits for an input gradient (or the head) that
    # wrote its output gradient or a later one
    dws = [c for c in prog.calls if c.label.endswith(".dW")]
    assert all(len(c.deps) == 1 for c in dws)


def _timed_call(fn, use_hook):
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    if use_hook:
        fg.profile_next_launch(k0, k1)
    fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1), (k0.elapsed_time(k1) if use_hook else None)


def test_profiling_events_bracket_the_main_kernel_only():
    """A split kernel gradient (main kernel + reduction): the library's
    events lie inside the call's and measure less than it; the hook is
    one-shot (a second call leaves the events where they were)."""
    shape = (1, 77, 79, 512, 512, 3, 1, 1)
    n, h, w, c, k, r, st, pd = shape
    d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
    assert fg.kernel_name(d, fg.OP_BWD_WEIGHT) == "wgrad_dma_kernel<true>"
    rng = np.random.default_rng(61)
    p, q = fg.out_dims(d)
    x = dev(synth.uniform(rng, (n, h, w, c)))
    dy = dev(synth.uniform(rng, (n, p, q, k)))
    dw = empty16((k, r, r, c))
    ws = workspace(d, fg.OP_BWD_WEIGHT)
    call = lambda: fg.conv2d_bwd_weight(d, x, dy, dw, ws)
    for _ in range(3):
        call()
    ratios = []
    for _ in range(5):
        t_call, t_main = _timed_call(call, True)
        assert 0 < t_main < t_call
        ratios.append(t_main / t_call)
    assert max(ratios) < 1.0
    # one-shot: the next call records nothing into the same events
    k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    fg.profile_next_launch(k0, k1)
    call()
    torch.cuda.synchronize()
    first = k0.elapsed_time(k1)
    call()
    torch.cuda.synchronize()
    assert k0.elapsed_time(k1) == first


def test_flags_clear_zeroes_exactly_its_range():
    base = torch.full((1000,), 7, dtype=torch.int32, device="cuda")
    fg.grad_flags_clear(base[3:700])
    got = host(base)
    assert (got[3:700] == 0).all() and (got[:3] == 7).all() and (got[700:] == 7).all()
