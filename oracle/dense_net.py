"""FC-DenseNet variant forward/backward on the oracle — TEST INFRASTRUCTURE
ONLY.

The network of Section 6.2 (dense blocks with growth rate 256, average
pooling, Huber loss), in the Tiramisu shape that ``synth.densenet_layers``
tabulates: stem conv; down levels of [dense block, 1x1 transition conv,
2x2 average pooling]; a bottleneck block; up levels of [4x4 stride-2
transposed conv of the previous block's new features, concatenation with
the skip (the down level's full concatenation), dense block]; a 1x1 head
over the last block's new features. A dense layer reads the concatenation
of its block's input and the outputs of the block's earlier layers; a ReLU
follows every layer except the head.

Each convolution is the oracle's fp64 evaluation; with ``store_fp16`` every
stored tensor (activations, pooled maps, gradients, and each partial sum of
a gradient that several consumers add into) is rounded once to fp16, as the
network stores it; otherwise everything stays in fp64. The backward pass
adds gradient contributions in this order: within a block, from the last
layer to the first; a down level's concatenation receives the transition
conv's input gradient first, then the skip gradient.
"""
import numpy as np

from . import conv2d_bwd_data, conv2d_bwd_weight, conv2d_fwd, conv_transpose2d_fwd
from . import dense as _dense


def _net(layers):
    by = {L.name: L for L in layers}
    levels = sum(1 for L in layers if L.name.startswith("TD"))
    per = sum(1 for L in layers if L.name.startswith("B."))
    return by, levels, per


class _Store:
    def __init__(self, fp16):
        self.fp16 = fp16

    def __call__(self, a):
        a = np.asarray(a, dtype=np.float64)
        return a.astype(np.float16) if self.fp16 else a

    def relu(self, a):
        return self(np.maximum(np.asarray(a, np.float64), 0.0))


def _gate(d, act):
    return np.where(np.asarray(act, np.float64) > 0, np.asarray(d, np.float64), 0.0)


def forward(layers, x16, weights, store_fp16=True):
    """Returns a dict: every layer's (post-ReLU) output under its name, the
    pooled maps 'P1'.., the skips 'skip1'.., every block's concatenations
    ('Z:<block>:<l>', l = 0 the block input) and 'y' (the head output)."""
    by, levels, per = _net(layers)
    W = {L.name: w for L, w in zip(layers, weights)}
    S = _Store(store_fp16)
    x = x16 if store_fp16 else np.asarray(x16, np.float64)
    out = {}

    def conv(name, inp, relu=True):
        L = by[name]
        if L.kind == "conv":
            r = conv2d_fwd(inp, W[name], L.stride, L.pad)
        else:
            r = conv_transpose2d_fwd(inp, W[name], L.stride, L.pad)
        return S.relu(r) if relu else S(r)

    def block(blk, z):
        out[f"Z:{blk}:0"] = z
        for l in range(1, per + 1):
            y = conv(f"{blk}.{l}", z)
            out[f"{blk}.{l}"] = y
            z = np.concatenate([z, y], axis=-1)
            out[f"Z:{blk}:{l}"] = z
        return z

    a = conv("C0", x)
    out["C0"] = a
    for d in range(1, levels + 1):
        z = block(f"D{d}", a)
        out[f"skip{d}"] = z
        t = conv(f"TD{d}", z)
        out[f"TD{d}"] = t
        a = _dense.avg_pool2d_fwd(t) if store_fp16 else \
            np.asarray(t).reshape(t.shape[0], t.shape[1] // 2, 2, t.shape[2] // 2, 2,
                                  t.shape[3]).mean(axis=(2, 4))
        out[f"P{d}"] = a
    c0 = a.shape[-1]
    z = block("B", a)
    nf = z[..., c0:]
    for d in range(levels, 0, -1):
        out[f"in:TU{d}"] = nf
        u = conv(f"TU{d}", nf)
        out[f"TU{d}"] = u
        z0 = np.concatenate([u, out[f"skip{d}"]], axis=-1)
        c0 = z0.shape[-1]
        z = block(f"U{d}", z0)
        nf = z[..., c0:]
    out["in:F1x1"] = nf
    out["y"] = conv("F1x1", nf, relu=False)
    return out


def backward(layers, fwd, x16, weights, g_out, store_fp16=True):
    """fp16 (or fp64) kernel gradients by layer name and the gradient of the
    network input, from the gradient g_out of the head output."""
    by, levels, per = _net(layers)
    W = {L.name: w for L, w in zip(layers, weights)}
    S = _Store(store_fp16)
    x = x16 if store_fp16 else np.asarray(x16, np.float64)
    k = by["D1.1"].y_shape[3]
    dW = {}

    def back(name, inp, dy):
        L = by[name]
        if L.kind == "conv":
            dW[name] = S(conv2d_bwd_weight(inp, dy, L.r, L.s, L.stride, L.pad))
            return S(conv2d_bwd_data(dy, W[name], inp.shape, L.stride, L.pad))
        dW[name] = S(conv2d_bwd_weight(dy, inp, L.r, L.s, L.stride, L.pad))
        return S(conv2d_fwd(dy, W[name], L.stride, L.pad))

    def block_back(blk, G):
        """G: gradient of the block's last concatenation (modified); returns
        it with the block input's gradient in its first channels."""
        c0 = fwd[f"Z:{blk}:0"].shape[-1]
        for l in range(per, 0, -1):
            name = f"{blk}.{l}"
            lo = c0 + (l - 1) * k
            dy = S(_gate(G[..., lo:lo + k], fwd[name]))
            dz = back(name, fwd[f"Z:{blk}:{l - 1}"], dy)
            G[..., :lo] = S(G[..., :lo].astype(np.float64) + np.asarray(dz, np.float64))
        return G

    def fresh(blk, dnew):
        zl = fwd[f"Z:{blk}:{per}"]
        G = np.zeros(zl.shape, dtype=np.float16 if store_fp16 else np.float64)
        G[..., zl.shape[-1] - dnew.shape[-1]:] = dnew
        return G

    dnf = back("F1x1", fwd["in:F1x1"], g_out)
    up = {}
    for d in range(1, levels + 1):
        G = block_back(f"U{d}", fresh(f"U{d}", dnf))
        nk = fwd[f"TU{d}"].shape[-1]
        du = S(_gate(G[..., :nk], fwd[f"TU{d}"]))
        dnf = back(f"TU{d}", fwd[f"in:TU{d}"], du)
        up[d] = G[..., nk:nk + fwd[f"skip{d}"].shape[-1]]
    G = block_back("B", fresh("B", dnf))
    dp = G[..., :fwd["Z:B:0"].shape[-1]]
    for d in range(levels, 0, -1):
        t = fwd[f"TD{d}"]
        if store_fp16:
            dt = _dense.avg_pool2d_bwd(dp, t)
        else:
            dt = _gate(np.repeat(np.repeat(np.asarray(dp) / 4.0, 2, axis=1), 2, axis=2), t)
        G = back(f"TD{d}", fwd[f"skip{d}"], dt)
        G = S(np.asarray(G, np.float64) + np.asarray(up[d], np.float64))
        G = block_back(f"D{d}", G)
        dp = G[..., :fwd[f"Z:D{d}:0"].shape[-1]]
    dc0 = S(_gate(dp, fwd["C0"]))
    dX = back("C0", x, dc0)
    return dW, dX
