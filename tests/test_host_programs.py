"""Host logic of the prepared step programs (no GPU): their stream
assignment and dependencies, built from CPU tensors with the CUDA stream
and event objects replaced by stand-ins (nothing is launched).

Chain step program: every kernel gradient waits for the call that wrote its
output gradient; the gradient path of a group waits for its last kernel
gradient; with an optimizer, every norms pass precedes every apply, layer
0's apply waits for the main stream's last call, each forward layer waits
for its own layer's apply of the previous run, the flag copy precedes the
applies, and the main stream's end-of-step wait leaves out the per-layer
applies. Dense network program: kernel gradients wait for their producer;
copy-stream calls wait for a main-stream call of the same step.
"""
import numpy as np
import pytest
import torch

import synth
from paper_1909_11150_amd import fcn
from paper_1909_11150_amd.densenet import DenseNet
from paper_1909_11150_amd.fcn import AdamLARS, Chain, LossScaler


class _Stream:
    cuda_stream = 0

    def __init__(self, *a, **k):
        pass


class _Event:
    def __init__(self, *a, **k):
        pass


@pytest.fixture
def no_cuda(monkeypatch):
    monkeypatch.setattr(torch.cuda, "current_stream", lambda *a, **k: _Stream())
    monkeypatch.setattr(torch.cuda, "Stream", _Stream)
    monkeypatch.setattr(torch.cuda, "Event", _Event)
    zeros = torch.zeros

    def zeros_unpinned(*a, **k):   # pinned host memory needs a device
        k.pop("pin_memory", None)
        return zeros(*a, **k)
    monkeypatch.setattr(torch, "zeros", zeros_unpinned)


def _chain(zero_copy, optimizer):
    layers = synth.fcn_layers(n=1, h=64, c_in=32, widths=(32, 64, 64, 64),
                              dec=(64, 64, 32, 32))
    w = [torch.zeros(L.w_shape, dtype=torch.float16) for L in layers]
    x = torch.zeros(layers[0].x_shape, dtype=torch.float16)
    kw = dict(optimizer=AdamLARS(), scaler=LossScaler()) if optimizer else {}
    return Chain(layers, w, x, device="cpu", group_cap_bytes=64 * 1024,
                 zero_copy=zero_copy, **kw)


def _common(calls):
    for i, c in enumerate(calls):
        assert all(d < i for d in c.deps), c.label          # producers come first
        assert all(calls[d].sid != c.sid for d in c.deps), c.label
        assert all(p > i for p in c.prev_deps), c.label     # previous run's calls


@pytest.mark.parametrize("zero_copy", [False, True])
@pytest.mark.parametrize("optimizer", [False, True])
def test_chain_program_dependencies(no_cuda, zero_copy, optimizer):
    ch = _chain(zero_copy, optimizer)
    t = torch.zeros(ch.layers[-1].y_shape, dtype=torch.float32)
    prog = ch.program(t, streams=3)
    calls = prog.calls
    _common(calls)
    idx = {c.label: i for i, c in enumerate(calls)}
    nl = len(ch.layers)
    for i, L in enumerate(ch.layers):
        dw = calls[idx[f"{L.name}.dW"]]
        assert dw.sid == 1
        # the output gradient's writer: the head for the last layer, else
        # the input gradient of the layer above
        writer = idx["head_grad"] if i == nl - 1 else idx[f"{ch.layers[i + 1].name}.dx"]
        assert dw.deps == (writer,)
    for gi, g in enumerate(ch.groups):
        first = [c for c in calls if c.label.startswith(f"G{gi}.")][0]
        last_dw = idx[f"{ch.layers[g['members'][-1]].name}.dW"]
        assert first.sid == 2 and first.deps == (last_dw,)
        labels = [c.label for c in calls if c.label.startswith(f"G{gi}.")]
        assert any(l.endswith(".unscale") for l in labels) == (not (zero_copy and optimizer))
    if not optimizer:
        assert not any(c.label.endswith(".apply") for c in calls)
        assert set(prog.step_final) == set(prog.final)
        return
    norms = [i for i, c in enumerate(calls) if c.label.endswith(".norms")]
    applies = {L.name: idx[f"{L.name}.apply"] for L in ch.layers}
    assert len(norms) == len(ch.groups)
    assert max(norms) < min(applies.values())
    assert idx["flags.copy"] < min(applies.values())
    a0 = calls[applies[ch.layers[0].name]]
    assert a0.sid == 1 and idx[f"{ch.layers[0].name}.dx"] in a0.deps
    for L in ch.layers:
        assert calls[idx[f"{L.name}.fwd"]].prev_deps == (applies[L.name],)
    # the end-of-step wait leaves the stream-2 applies to the next forward pass
    assert all(calls[j].sid != 2 for j in prog.step_final)


def test_dense_program_dependencies(no_cuda):
    layers = synth.densenet_layers(n=1, h=32, c_in=32, c0=32, growth=32, levels=2,
                                   per_block=2)
    w = [torch.zeros(L.w_shape, dtype=torch.float16) for L in layers]
    x = torch.zeros(layers[0].x_shape, dtype=torch.float16)
    net = DenseNet(layers, w, x, device="cpu")
    t = torch.zeros(layers[-1].y_shape, dtype=torch.float32)
    for streams in (1, 2, 3):
        prog = net.program(t, streams=streams)
        calls = prog.calls
        _common(calls)
        assert len(prog.streams) == streams
        for i, c in enumerate(calls):
            if c.sid == 1:
                assert c.label.endswith(".dW") and c.deps == (i - 1,)
            if c.sid == 2:
                assert c.label.endswith(".new"), c.label
                assert any(calls[d].sid == 0 for d in c.deps), c.label
        if streams == 1:
            assert all(c.sid == 0 and not c.deps for c in calls)
        # every conv layer appears with its three passes
        labels = {c.label for c in calls}
        for L in layers:
            assert {f"{L.name}.fwd", f"{L.name}.dW", f"{L.name}.dx"} <= labels


def _elements(sl, npix):
    """Element offsets (in the slice's buffer) of a slice over npix pixels."""
    return (sl.off + np.arange(npix)[:, None] * sl.ld + np.arange(sl.ch)[None, :]).ravel()


@pytest.mark.parametrize("per", [2, 3])
def test_dense_layout_concatenations_in_place(no_cuda, per):
    """The dense network's level buffers: each layer reads exactly the
    channels before its own output slice (its block input, then the earlier
    layers' outputs, in concatenation order); a down block's skip is its
    input and all its outputs; an up block's input is the transition-up
    output followed by the skip; no two outputs share an element."""
    layers = synth.densenet_layers(n=1, h=16, c_in=16, c0=16, growth=8, levels=2,
                                   per_block=per)
    w = [torch.zeros(L.w_shape, dtype=torch.float16) for L in layers]
    x = torch.zeros(layers[0].x_shape, dtype=torch.float16)
    net = DenseNet(layers, w, x, device="cpu")
    k, nk = net.k, per * net.k
    for blk in net._blocks():
        c0 = net.L[f"{blk}.1"].x_shape[3]
        for l in range(1, per + 1):
            name = f"{blk}.{l}"
            i, o = net.inp[name], net.out[name]
            assert i.off + i.ch == o.off or (not blk.startswith("D") and l == per)
            assert i.ch == c0 + (l - 1) * k == net.L[name].x_shape[3]
            if l < per or blk.startswith("D"):
                assert o.t is i.t and o.ld == i.ld and o.ch == k
            else:     # a bottleneck or up block's last layer: its new features
                assert o.t is net.NF[blk] and o.off == (per - 1) * k
    for d in (1, 2):
        z = net.Z[f"U{d}"]
        skip = net.inp[f"TD{d}"]
        assert skip.t is z and skip.off == nk and skip.off == net.out[f"TU{d}"].ch
        assert skip.ch == net.inp[f"D{d}.1"].ch + per * k
        assert net.inp[f"D{d}.1"].off == nk
        assert net.inp[f"U{d}.1"].off == 0 and net.inp[f"U{d}.1"].ch == nk + skip.ch
    assert net.out["C0"] == net.inp["D1.1"]
    # outputs are pairwise disjoint, buffer by buffer
    seen = {}
    for name, sl in net.out.items():
        L = net.L[name]
        e = _elements(sl, L.y_shape[0] * L.y_shape[1] * L.y_shape[2])
        assert e.max() < sl.t.numel()
        key = sl.t.data_ptr()
        prev = seen.setdefault(key, np.zeros(sl.t.numel(), bool))
        assert not prev[e].any(), name
        prev[e] = True


def test_dense_program_gradient_groups(no_cuda):
    """Each group's pack, unscale and unpack follow every member's kernel
    gradient on the kernel-gradient stream; the flags are cleared first."""
    layers = synth.densenet_layers(n=1, h=32, c_in=32, c0=32, growth=32, levels=2,
                                   per_block=2)
    w = [torch.zeros(L.w_shape, dtype=torch.float16) for L in layers]
    x = torch.zeros(layers[0].x_shape, dtype=torch.float16)
    net = DenseNet(layers, w, x, device="cpu", group_cap_bytes=48 * 1024)
    t = torch.zeros(layers[-1].y_shape, dtype=torch.float32)
    for streams in (1, 2):
        calls = net.program(t, streams=streams).calls
        idx = {c.label: i for i, c in enumerate(calls)}
        side = 1 if streams > 1 else 0
        first_side = min(i for i, c in enumerate(calls) if c.sid == side)
        assert calls[first_side].label == "flags.clear" or side == 0
        assert idx["flags.clear"] < min(idx[f"{m}.dW"] for m in net.dw_order())
        for gi, g in enumerate(net.groups):
            p, u, q = idx[f"G{gi}.pack"], idx[f"G{gi}.unscale"], idx[f"G{gi}.unpack"]
            assert p < u < q and all(calls[j].sid == side for j in (p, u, q))
            assert max(idx[f"{m}.dW"] for m in g["members"]) < p
            assert all(calls[idx[f"{m}.dW"]].sid == side for m in g["members"])
