"""A CPU stand-in for the library's calls, built from the oracle — TEST
INFRASTRUCTURE ONLY (the product has no CPU path; this module lives with the
tests and only tests install it).

Each function has the signature of the binding's function of the same name
and writes its result into the given (CPU) output tensor: convolutions are
the oracle's fp64 values with the call's epilogue, rounded once to fp16; the
gradient path is the oracle's pack, unscale-with-check and unpack. With
these in place of the binding's calls, the encoder-decoder driver's eager
step runs on the CPU, so its wiring (descriptors, operand roles, gates,
group offsets) can be checked against the oracle's own chain.
"""
import numpy as np
import torch

import oracle
import paper_1909_11150_amd as fg
from oracle import grad as G

NAMES = ("conv2d_fwd", "conv_transpose2d_fwd", "conv2d_bwd_data", "conv2d_bwd_weight",
         "l2_head_grad", "grad_group_pack", "grad_unscale_check", "grad_group_unpack")


def _np(t):
    return t.detach().cpu().numpy()


def _put(out, a):
    out.copy_(torch.from_numpy(np.ascontiguousarray(a)).reshape(out.shape))


def _epi(epi):
    return {fg.EPI_NONE: None, fg.EPI_RELU: "relu", fg.EPI_GATE: "gate"}[epi]


def _gate(g):
    return None if g is None else _np(g)


def _equal_strides(d):
    assert d.stride_h == d.stride_w and d.pad_h == d.pad_w and not d.x_ld and not d.y_ld


def conv2d_fwd(desc, x, w, y, epi=fg.EPI_NONE, gate=None, ws=None, stream=None):
    _equal_strides(desc)
    r = oracle.conv2d_fwd(_np(x), _np(w), desc.stride_h, desc.pad_h, epi=_epi(epi),
                          gate=_gate(gate))
    _put(y, r.astype(np.float16))


def conv_transpose2d_fwd(desc, x, w, y, epi=fg.EPI_NONE, gate=None, ws=None, stream=None):
    _equal_strides(desc)
    r = oracle.conv_transpose2d_fwd(_np(x), _np(w), desc.stride_h, desc.pad_h,
                                    epi=_epi(epi), gate=_gate(gate))
    _put(y, r.astype(np.float16))


def conv2d_bwd_data(desc, dy, w, dx, epi=fg.EPI_NONE, gate=None, ws=None, stream=None):
    _equal_strides(desc)
    r = oracle.conv2d_bwd_data(_np(dy), _np(w), tuple(dx.shape), desc.stride_h, desc.pad_h,
                               epi=_epi(epi), gate=_gate(gate))
    _put(dx, r.astype(np.float16))


def conv2d_bwd_weight(desc, x, dy, dw, ws=None, stream=None):
    _equal_strides(desc)
    r = oracle.conv2d_bwd_weight(_np(x), _np(dy), desc.r, desc.s, desc.stride_h, desc.pad_h)
    _put(dw, r.astype(np.float16))


def l2_head_grad(y, t, scale, dy, stream=None):
    yv = _np(y).astype(np.float64)
    tv = _np(t).astype(np.float64)
    with np.errstate(over="ignore"):
        _put(dy, (np.float64(scale) * (yv - tv)).astype(np.float16))


def grad_group_pack(srcs, offsets, group, stream=None):
    grp = {"members": list(range(len(srcs))), "offsets": list(offsets),
           "numel": group.numel()}
    bits = G.pack([_np(s).view(np.uint16).ravel() for s in srcs], grp)
    _put(group, bits.view(np.float16))


def grad_unscale_check(group, inv_scale, out_f32, flag, numel=None, stream=None):
    r32, found = G.unscale_check(_np(group).view(np.uint16), np.float32(inv_scale))
    _put(out_f32, r32)
    if found:
        flag[0] = 1


def grad_group_unpack(group_f32, dsts, offsets, stream=None):
    g = _np(group_f32)
    for d, off in zip(dsts, offsets):
        _put(d, g[off:off + d.numel()])
