"""The encoder-decoder driver's eager step on the CPU, with every library
call replaced by the oracle-backed stand-in of tests/fake_backend.py (the
"fake backend" a test of the harness can run without a GPU).

The driver's own wiring then decides everything: which descriptor each pass
gets (including the transposed convolutions' adjoint passes and their
operand roles), which epilogue and gate, the order of the backward pass, the
gradient groups the library's planner forms and the offsets the group path
uses. The test runs forward, loss-scaled head gradient and backward with the
grouped gradient path on a reduced network and requires every activation,
input gradient, kernel gradient, group buffer, fp32 master gradient and flag
to equal, bit for bit, the oracle's own chain (oracle/chain.py, fp16 storage
at layer boundaries) and its gradient path (oracle/grad.py) (Section 5.2:
three passes per layer; Section 4.2 Grouping; Section 6.2 loss scaling).
"""
import numpy as np
import pytest
import torch

import fake_backend
import synth
from oracle import chain as OC
from oracle import grad as G
from paper_1909_11150_amd import fcn
from paper_1909_11150_amd.fcn import Chain

S = 2.0 ** 15


@pytest.fixture
def fake(monkeypatch):
    for name in fake_backend.NAMES:
        monkeypatch.setattr(fcn, name, getattr(fake_backend, name))


def _bits(a):
    return np.ascontiguousarray(a).view(np.uint16)


@pytest.mark.parametrize("inject", [False, True])
def test_eager_step_wiring_matches_the_oracle_chain(fake, inject):
    layers = synth.fcn_layers(n=1, h=32, c_in=16, widths=(16, 32, 32, 32),
                              dec=(32, 32, 16, 16))
    x = synth.diffraction_like(1, 32, 16, seed=0)
    w = synth.he_weights(layers, seed=1)
    t = synth.smooth_target(1, 32, seed=4)
    ch = Chain(layers, w, x, device="cpu", loss_scale=S, group_cap_bytes=16 * 1024)
    assert len(ch.groups) > 2  # several groups, some with several members
    ch.forward()
    ch.head_grad(torch.from_numpy(t))
    if inject:  # a non-finite output gradient: every group downstream flags
        ch.g[-1].view(-1)[7] = float("inf")
    ch.backward(grad_path=True)

    acts = OC.forward(layers, x, w)
    for i in range(len(layers)):
        assert np.array_equal(_bits(ch.acts[i + 1].numpy()), _bits(acts[i + 1])), layers[i].name
    head = OC.head_grad(acts[-1], t, S)
    if inject:
        head = head.copy()
        head.reshape(-1)[7] = np.inf
    assert np.array_equal(_bits(ch.g[-1].numpy()), _bits(head))
    with np.errstate(invalid="ignore", over="ignore"):
        dws, dxs = OC.backward(layers, acts, w, head)
    for i, L in enumerate(layers):
        assert np.array_equal(_bits(ch.dw[i].numpy()), _bits(dws[i])), f"{L.name} dW"
        assert np.array_equal(_bits(ch.g[i].numpy()), _bits(dxs[i])), f"{L.name} dx"

    numels = [a.size for a in w]
    flags = ch.flags.numpy()
    for gi, grp in enumerate(ch.groups):
        ref16 = G.pack([_bits(d).ravel() for d in dws], grp)
        assert np.array_equal(_bits(ch.gbuf16[gi].numpy()), ref16), f"group {gi}"
        r32, found = G.unscale_check(ref16, np.float32(1.0 / S))
        assert int(flags[gi]) == int(found), f"group {gi} flag"
        got32 = ch.gbuf32[gi].numpy()
        fin = np.isfinite(r32)
        assert np.array_equal(got32[fin].view(np.uint32), r32[fin].view(np.uint32))
        assert np.array_equal(np.isnan(got32), np.isnan(r32))
        for m, v in G.unpack(r32, grp, numels).items():
            got = ch.master[m].numpy().ravel()
            assert np.array_equal(np.isnan(got), np.isnan(v)), f"master {m}"
            assert np.array_equal(got[np.isfinite(v)].view(np.uint32),
                                  v[np.isfinite(v)].view(np.uint32)), f"master {m}"
    if inject:
        assert flags.any()
    else:
        assert not flags.any()
