"""GPU tests of the full training step (Section 6.2): the reduced
encoder-decoder with gradient groups, the layer-wise adaptive Adam update of
fp32 master weights and the backoff loss scale, run by the step program.

Each step is checked against the oracle on the GPU's own inputs of that
step: the head gradient against fp16(2 S (y - t) / numel) with the scale S
the step was given (bit for bit: both round one fp64 value), the unpacked
gradients against fp16 dW / S (exact; with zero-copy groups the optimizer
reads dW / S from the fp16 slots itself), the group flags against the
non-finite entries of dW, a skipped step against the state before it (bit
for bit), an applied step layer by layer against the optimizer oracle (the
rule of the optimizer's own parity tests), and the loss-scale sequence
against the oracle's backoff rule. The three-stream program must give the
same bits as the one-stream order.
"""
import numpy as np
import pytest
import torch

import synth
from gpu_util import OPT_HP, check_opt_layer, dev, host
from oracle import optim as O
from paper_1909_11150_amd.fcn import AdamLARS, Chain, LossScaler, LRSchedule

pytestmark = pytest.mark.gpu

CAP = 64 * 1024


def _reduced():
    layers = synth.fcn_layers(n=1, h=64, c_in=32, widths=(32, 64, 64, 64),
                              dec=(64, 64, 32, 32))
    x = synth.diffraction_like(1, 64, 32, seed=0)
    w = synth.he_weights(layers, seed=1)
    t = synth.smooth_target(1, 64, seed=4)
    return layers, x, w, t


def _opt(lr):
    return AdamLARS(lr=lr, **OPT_HP)


def _state(ch):
    torch.cuda.synchronize()
    c = lambda ts: [x.detach().cpu().numpy().ravel().copy() for x in ts]
    return dict(w32=c(ch.w32), m=c(ch.m), v=c(ch.v), w16=c(ch.w),
                step=int(ch.step_count.item()))


def _same(a, b):
    for k in ("w32", "m", "v", "w16"):
        for x, y in zip(a[k], b[k]):
            if not np.array_equal(x.view(np.uint8), y.view(np.uint8)):
                return False
    return a["step"] == b["step"]


def _run(ch, t, nsteps, lr_of, program=None):
    """Run nsteps steps, checking each against the oracle; returns the
    sequence of (scale, found)."""
    prog = program if program is not None else ch.program(t)
    td = host(t).astype(np.float64).ravel()
    seq = []
    for _ in range(nsteps):
        ch.observe()
        S = ch.loss_scale
        applied_before = ch.applied
        before = _state(ch)
        prog.run()
        ch.observe()
        found = ch.last_found
        after = _state(ch)
        # head gradient with this step's scale
        y = host(ch.acts[-1]).astype(np.float64).ravel()
        with np.errstate(over="ignore"):  # overflow to +-inf is the case tested
            ref = (2.0 * S / y.size * (y - td)).astype(np.float16)
        np.testing.assert_array_equal(host(ch.g[-1]).ravel().view(np.uint16),
                                      ref.view(np.uint16))
        # unpacked gradients, flags
        dws = [host(d).ravel() for d in ch.dw]
        inv = np.float32(1.0 / S)
        if ch.zero_copy:  # the optimizer reads the fp16 slots: dW / S
            gs = [d.astype(np.float32) * inv for d in dws]
        else:
            gs = [host(m).ravel() for m in ch.master]
            for d, g in zip(dws, gs):
                np.testing.assert_array_equal(g, d.astype(np.float32) * inv)
        assert found == any(not np.isfinite(d.astype(np.float32)).all() for d in dws)
        if found:
            assert _same(before, after), "a flagged step changed the state"
            assert ch.applied == applied_before
        else:
            tstep = before["step"] + 1
            assert after["step"] == tstep == ch.applied == applied_before + 1
            lr = lr_of(applied_before)
            for i in range(len(ch.layers)):
                check_opt_layer(before["w32"][i], before["m"][i], before["v"][i],
                                gs[i], tstep, lr, after["w32"][i], after["m"][i],
                                after["v"][i], after["w16"][i])
        seq.append((S, found))
    return seq


def test_steps_update_the_master_weights():
    """Three clean steps at a fixed scale under a warm-up schedule."""
    layers, x, w, t = _reduced()
    sch = LRSchedule(1e-4, 4e-4, warmup=2)
    ch = Chain(layers, w, x, loss_scale=2.0 ** 10, group_cap_bytes=CAP,
               optimizer=_opt(sch))
    assert len(ch.groups) > 1
    w16_0 = [np.asarray(a) for a in w]
    np.testing.assert_array_equal(_state(ch)["w32"][3], w16_0[3].astype(np.float32).ravel())
    seq = _run(ch, dev(t), 3, sch)
    assert [f for _, f in seq] == [False] * 3
    assert ch.applied == 3
    # the forward pass reads the updated fp16 weights
    assert not np.array_equal(host(ch.w[0]), w16_0[0])


@pytest.mark.parametrize("zero_copy", [False, True])
def test_overflow_backs_off_and_skips(zero_copy):
    """A target far from the output overflows the head gradient and the
    kernel gradients at the initial scale: those steps are skipped and the
    scale backs off until the gradients fit, then grows again after
    `interval` clean steps."""
    layers, x, w, t = _reduced()
    t = t - np.float32(6000.0)
    sc = LossScaler(2.0 ** 15, interval=3)
    ch = Chain(layers, w, x, group_cap_bytes=CAP, zero_copy=zero_copy,
               optimizer=_opt(1e-3), scaler=sc)
    seq = _run(ch, dev(t), 24, lambda k: 1e-3)
    print("scale, found:", seq)
    found = [f for _, f in seq]
    assert found[0] and found[1] and not all(found), found
    s, c = 2.0 ** 15, 0
    for S, f in seq:
        assert S == s
        s, c, _ = O.loss_scale_next(s, c, f, 3)
    assert (sc.scale, sc.clean) == (s, c)
    assert ch.applied == found.count(False)
    assert any(b > a for (a, _), (b, _) in zip(seq, seq[1:])), "the scale never grew"


def test_fp16_slot_optimizer_equals_fp32_gradient_path():
    """Zero-copy groups (optimizer on the fp16 slots, no unscale/unpack) and
    packed groups (optimizer on the unpacked fp32 gradients) give the same
    bits over steps with skips and scale changes."""
    layers, x, w, t = _reduced()
    td = dev(t - np.float32(40.0))
    out = []
    for zc in (False, True):
        ch = Chain(layers, w, x, group_cap_bytes=CAP, zero_copy=zc,
                   optimizer=_opt(1e-3), scaler=LossScaler(2.0 ** 15, interval=2))
        prog = ch.program(td)
        labels = [c.label for c in prog.calls]
        assert any(".norms" in c for c in labels)
        assert any(".unscale" in c for c in labels) == (not zc)
        for _ in range(8):
            prog.run()
        ch.observe()
        out.append((_state(ch), ch.loss_scale, ch.applied))
    assert _same(out[0][0], out[1][0])
    assert out[0][1:] == out[1][1:]


@pytest.mark.parametrize("zero_copy", [False, True])
def test_three_streams_match_one_stream(zero_copy):
    layers, x, w, t = _reduced()
    t = t - np.float32(40.0)
    td = dev(t)
    out = []
    for streams in (3, 1):
        ch = Chain(layers, w, x, group_cap_bytes=CAP, zero_copy=zero_copy,
                   optimizer=_opt(LRSchedule(1e-4, 1e-3, warmup=3)),
                   scaler=LossScaler(2.0 ** 15, interval=2))
        prog = ch.program(td, streams=streams)
        for _ in range(6):
            prog.run()
        ch.observe()
        out.append((_state(ch), ch.loss_scale, ch.applied))
    assert _same(out[0][0], out[1][0])
    assert out[0][1:] == out[1][1:]
    assert out[0][2] > 0
