"""An independent fp32-accumulating run of the network chain (PyTorch CPU
float32 convolutions, activations and gradients stored in fp16 after every
layer, ReLU gating by the stored activations). Used only to calibrate how far
any correct fp32-accumulating implementation drifts from the fp64 oracle
chain; it is not a reference the GPU is compared against."""
import numpy as np
import torch
import torch.nn.functional as F


def _nchw(a):
    return torch.from_numpy(np.ascontiguousarray(
        np.asarray(a, np.float32).transpose(0, 3, 1, 2)))


def _nhwc(t):
    return t.detach().numpy().transpose(0, 2, 3, 1)


def _w(w16):
    return torch.from_numpy(np.ascontiguousarray(
        w16.astype(np.float32).transpose(0, 3, 1, 2)))


def _f16(a):
    return np.asarray(a, np.float32).astype(np.float16)


def _apply(L, x, w):
    if L.kind == "conv":
        return F.conv2d(x, w, stride=L.stride, padding=L.pad)
    return F.conv_transpose2d(x, w, stride=L.stride, padding=L.pad)


def forward(layers, x16, weights):
    acts = [x16]
    for L, w in zip(layers, weights):
        with torch.no_grad():
            y = _nhwc(_apply(L, _nchw(acts[-1]), _w(w)))
        acts.append(_f16(np.maximum(y, 0) if L.relu else y))
    return acts


def backward(layers, acts, weights, dy16):
    dws, dxs = [None] * len(layers), [None] * len(layers)
    d = dy16
    for i in reversed(range(len(layers))):
        L = layers[i]
        xt = _nchw(acts[i]).requires_grad_(True)
        wt = _w(weights[i]).requires_grad_(True)
        _apply(L, xt, wt).backward(_nchw(d))
        dx = _nhwc(xt.grad)
        if i > 0 and layers[i - 1].relu:
            dx = np.where(acts[i].astype(np.float32) > 0, dx, 0.0)
        dxs[i] = _f16(dx)
        dws[i] = _f16(wt.grad.numpy().transpose(0, 2, 3, 1))
        d = dxs[i]
    return dws, dxs
