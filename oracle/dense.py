"""Glue of the FC-DenseNet variant, plain NumPy — TEST INFRASTRUCTURE ONLY.

Section 6.2 (Neural Network Architecture) builds the network from dense
blocks whose layers' outputs are concatenated along the channels (growth
rate 256) and downsamples with average pooling instead of max pooling; the
loss (Model Implementation, the loss equation) is the Huber loss with a
cutoff delta. Each function below is the plain definition, evaluated in
fp64 on fp16 inputs (which fp64 holds exactly) and rounded once to fp16,
nearest-even, overflow to infinity (numpy's float64 -> float16 cast).

Readings:
  * Huber loss per output: d^2/2 for |d| <= delta, delta (|d| - delta/2)
    beyond; the network's loss is its mean over the outputs times the loss
    scale S, so the head gradient is S/numel * clamp(y - t, -delta, delta);
  * average pooling: 2 x 2 windows with stride 2 over even H and W;
  * concatenation: channels of the pieces in order, NHWC; its backward
    reads each piece's slice and sums the gradients that reach a slice.
"""
import numpy as np


def huber_head_grad(y16, target, scale, delta):
    """dy = fp16(scale * clamp(y - t, -delta, delta)), fp64, one rounding."""
    d = np.asarray(y16).astype(np.float64) - np.asarray(target).astype(np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        return (np.float64(scale) * np.clip(d, -delta, delta)).astype(np.float16)


def avg_pool2d_fwd(x16):
    """Mean of each 2 x 2 window (stride 2) of an N x H x W x C tensor."""
    x = np.asarray(x16).astype(np.float64)
    n, h, w, c = x.shape
    s = x.reshape(n, h // 2, 2, w // 2, 2, c).sum(axis=(2, 4))
    return (s / 4.0).astype(np.float16)


def avg_pool2d_bwd(dy16, gate16=None):
    """Each input of a window receives a quarter of the window's output
    gradient; zero where the gate (the pooled ReLU output) is <= 0."""
    dy = np.asarray(dy16).astype(np.float64) / 4.0
    dx = np.repeat(np.repeat(dy, 2, axis=1), 2, axis=2)
    if gate16 is not None:
        dx = np.where(np.asarray(gate16).astype(np.float64) > 0, dx, 0.0)
    return dx.astype(np.float16)


def channel_slice_copy(src16, dst16, gate16=None, accumulate=False):
    """src and dst: P x nch views (one row per pixel) of the slices. Returns
    the new dst slice: src (zero where gate <= 0), or fp16(dst + that)."""
    v = np.asarray(src16).astype(np.float64)
    if gate16 is not None:
        v = np.where(np.asarray(gate16).astype(np.float64) > 0, v, 0.0)
    if accumulate:
        with np.errstate(invalid="ignore", over="ignore"):
            v = np.asarray(dst16).astype(np.float64) + v
    with np.errstate(over="ignore"):
        return v.astype(np.float16)


def concat_channels(pieces16):
    """Dense concatenation: the pieces' channels in order (NHWC)."""
    return np.concatenate([np.asarray(p, np.float16) for p in pieces16], axis=-1)
