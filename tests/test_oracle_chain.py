"""Pin for the oracle's network chain (CPU only).

The chain's forward and backward passes (layer order, ReLU placement, the
gradient gating, the transposed-conv adjoints, the loss-scaled L2 head) are
checked against PyTorch float64 autograd of the same network. The oracle
stores every activation and gradient in fp16 while PyTorch does not, so the
two agree to the fp16 rounding budget, not exactly: a wrong gate, sign,
operand or layer order moves the result by O(1) relative error.
"""
import numpy as np
import torch
import torch.nn.functional as F

import synth
from oracle import chain


def _torch_net(layers, x16, weights, target, scale):
    x = torch.from_numpy(x16.astype(np.float64).transpose(0, 3, 1, 2).copy())
    ws = []
    for L, w in zip(layers, weights):
        wt = torch.from_numpy(w.astype(np.float64).transpose(0, 3, 1, 2).copy())
        ws.append(wt.requires_grad_(True))
    a = x
    for L, w in zip(layers, ws):
        if L.kind == "conv":
            a = F.conv2d(a, w, stride=L.stride, padding=L.pad)
        else:
            a = F.conv_transpose2d(a, w, stride=L.stride, padding=L.pad)
        if L.relu:
            a = torch.relu(a)
    t = torch.from_numpy(target.astype(np.float64).transpose(0, 3, 1, 2).copy())
    loss = scale * torch.mean((a - t) ** 2)
    loss.backward()
    y = a.detach().numpy().transpose(0, 2, 3, 1)
    return y, [w.grad.numpy().transpose(0, 2, 3, 1) for w in ws]


def _rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.linalg.norm(a - b) / np.linalg.norm(b)


def test_mini_fcn_chain_matches_torch_autograd(oracle_lib):
    layers = synth.fcn_layers(n=1, h=32, c_in=8, widths=(8, 16, 16, 16),
                              dec=(16, 16, 8, 8))
    x = synth.diffraction_like(1, 32, 8, seed=0)
    w = synth.he_weights(layers, seed=1)
    t = synth.smooth_target(1, 32, seed=4)
    scale = 2.0 ** 10
    acts = chain.forward(layers, x, w)
    dy = chain.head_grad(acts[-1], t, scale)
    dws, _ = chain.backward(layers, acts, w, dy)
    y_ref, dws_ref = _torch_net(layers, x, w, t, scale)
    assert _rel(acts[-1], y_ref) < 2e-2
    for L, a, b in zip(layers, dws, dws_ref):
        assert _rel(a, b) < 5e-2, L.name
