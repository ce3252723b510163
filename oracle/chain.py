"""Encoder-decoder forward/backward on the oracle — TEST INFRASTRUCTURE ONLY.

The chain follows the training step of the paper's fully convolutional
network (Section 6.2, Neural Network Architecture and Model Implementation):
each layer's output is stored in fp16 (the float16 implementation), a ReLU
follows every layer except the head, the loss gradient is scaled by the loss
scale before back-propagation, and every layer contributes its three
convolution passes (Section 5.2). Each convolution is evaluated in fp64 by
the oracle and rounded once to fp16 where the network stores it.

Transposed-conv backward passes are the adjoints of the transposed conv:
  dx = forward conv of dy with Wt read as a KRSC weight (K = C_in, C = C_out)
  dWt = weight gradient of that conv with the roles of x and dy exchanged.
"""
import numpy as np

from . import (conv2d_bwd_data, conv2d_bwd_weight, conv2d_fwd,
               conv_transpose2d_fwd)
from . import grad as _grad


def _f16(a):
    return np.asarray(a, dtype=np.float64).astype(np.float16)


def layer_forward(L, x16, w16):
    epi = "relu" if L.relu else None
    if L.kind == "conv":
        return conv2d_fwd(x16, w16, L.stride, L.pad, epi=epi)
    return conv_transpose2d_fwd(x16, w16, L.stride, L.pad, epi=epi)


def layer_backward(L, x16, w16, dy16, gate_input):
    """Return (dx fp64 or None, dW fp64). dy16 is the gradient w.r.t. the
    layer's pre-activation output; gate_input says whether x16 is itself a
    ReLU output, in which case dx is gated by x16 > 0."""
    epi = "gate" if gate_input else None
    if L.kind == "conv":
        dw = conv2d_bwd_weight(x16, dy16, L.r, L.s, L.stride, L.pad)
        dx = conv2d_bwd_data(dy16, w16, x16.shape, L.stride, L.pad, epi=epi,
                             gate=x16)
    else:
        dw = conv2d_bwd_weight(dy16, x16, L.r, L.s, L.stride, L.pad)
        dx = conv2d_fwd(dy16, w16, L.stride, L.pad, epi=epi, gate=x16)
    return dx, dw


def _store(a, fp16):
    return _f16(a) if fp16 else np.asarray(a, dtype=np.float64)


def forward(layers, x16, weights, store_fp16=True):
    """Activations [x, a1, ..., aL]; each a_i rounded once to fp16 (the
    network's storage format) unless store_fp16 is False, in which case the
    chain runs entirely in fp64 (used to measure what fp16 storage costs)."""
    acts = [x16 if store_fp16 else np.asarray(x16, dtype=np.float64)]
    for L, w in zip(layers, weights):
        acts.append(_store(layer_forward(L, acts[-1], w), store_fp16))
    return acts


def backward(layers, acts, weights, dy_out16, store_fp16=True):
    """fp16 weight gradients in forward order and fp16 input gradients.

    dy_out16 is the gradient w.r.t. the last layer's pre-activation output.
    Returns (dws, dxs) where dxs[i] is the gradient w.r.t. acts[i].
    """
    nl = len(layers)
    dws = [None] * nl
    dxs = [None] * nl
    dy = dy_out16
    for i in reversed(range(nl)):
        L = layers[i]
        gate = i > 0 and layers[i - 1].relu
        dx, dw = layer_backward(L, acts[i], weights[i], dy, gate)
        dws[i] = _store(dw, store_fp16)
        dxs[i] = _store(dx, store_fp16)
        dy = dxs[i]
    return dws, dxs


def head_grad(y16, target, loss_scale, store_fp16=True):
    if store_fp16:
        return _grad.head_grad(y16, target, loss_scale)
    y = np.asarray(y16, dtype=np.float64)
    return loss_scale * 2.0 * (y - np.asarray(target, np.float64)) / y.size
