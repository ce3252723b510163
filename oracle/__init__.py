"""CPU oracle for the fp16 FCN training-step hot path — TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. It shares no code with the HIP library and never calls
it; the product path must not import anything from here.

Contents
  conv2d_fwd / conv2d_bwd_data / conv2d_bwd_weight / conv_transpose2d_fwd
      fp64 direct-loop convolutions (``conv_oracle.c``) on fp16 inputs upcast
      exactly, with the ReLU / ReLU-gradient epilogues applied in fp64.
      The operation count of each is the paper's direct-convolution count
      (Section 5.2, equation OPS_conv); forward, kernel gradient and input
      gradient are the three passes of its performance definition (Section
      5.2, factor 3 in the Sustained/Peak equations).
  *_points
      the same definitions evaluated only at listed flat output indices, for
      checking full-size outputs by sampling.
  grad (module)
      group planner, fusion-buffer pack, loss-scale unscale with the
      non-finite check, and unpack (Section 4.2; Section 6.2 mixed precision
      with loss scaling).
  chain (module)
      the encoder-decoder forward and backward passes built from the above.
  optim (module)
      the layer-wise adaptive Adam update and the loss-scale backoff that
      consume the unpacked fp32 gradients (Section 6.2).
  dense (module)
      the FC-DenseNet variant's glue: Huber head gradient, 2 x 2 average
      pooling and its gradient, channel concatenation and slice copies
      (Section 6.2).
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(HERE, "liboracle_conv.so")
_lib = None

OP_FWD, OP_BWD_DATA, OP_BWD_WEIGHT, OP_CONVT = 0, 1, 2, 3


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        lib = ctypes.CDLL(_LIB_PATH)
        p64 = ctypes.POINTER(ctypes.c_int64)
        pd = ctypes.POINTER(ctypes.c_double)
        lib.oracle_conv_out_dims.argtypes = [p64, ctypes.c_int, p64]
        lib.oracle_conv_out_dims.restype = None
        lib.oracle_conv_full.argtypes = [p64, ctypes.c_int, pd, pd, pd]
        lib.oracle_conv_full.restype = None
        lib.oracle_conv_points.argtypes = [p64, ctypes.c_int, pd, pd,
                                           ctypes.c_int64, p64, pd]
        lib.oracle_conv_points.restype = None
        _lib = lib
    return _lib


def _f64(a):
    a = np.asarray(a)
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a, t=ctypes.c_double):
    return a.ctypes.data_as(ctypes.POINTER(t))


def _shape_vec(n, h, w, c, k, r, s, stride, pad):
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    return np.array([n, h, w, c, k, r, s, sh, sw, ph, pw], dtype=np.int64)


def out_dims(shape_vec, op):
    d = np.zeros(4, dtype=np.int64)
    _load().oracle_conv_out_dims(_ptr(shape_vec, ctypes.c_int64), op,
                                 _ptr(d, ctypes.c_int64))
    return tuple(int(v) for v in d)


def _run_full(shape_vec, op, a, b):
    a, b = _f64(a), _f64(b)
    d = out_dims(shape_vec, op)
    out = np.empty(d, dtype=np.float64)
    _load().oracle_conv_full(_ptr(shape_vec, ctypes.c_int64), op, _ptr(a),
                             _ptr(b), _ptr(out))
    return out


def _run_points(shape_vec, op, a, b, flat_idx):
    a, b = _f64(a), _f64(b)
    idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
    out = np.empty(idx.shape[0], dtype=np.float64)
    _load().oracle_conv_points(_ptr(shape_vec, ctypes.c_int64), op, _ptr(a),
                               _ptr(b), idx.shape[0],
                               _ptr(idx, ctypes.c_int64), _ptr(out))
    return out


# ---- epilogues (fused ReLU and ReLU-gradient of the FC network) ----------
def relu(acc):
    """ReLU after a convolution: positive values pass, everything else is +0."""
    return np.where(acc > 0, acc, 0.0)


def relu_grad(acc, gate):
    """ReLU backward: pass the gradient where the forward activation is > 0."""
    g = np.asarray(gate).astype(np.float64)
    return np.where(g > 0, acc, 0.0)


def _epilogue(acc, epi, gate):
    if epi in (None, "none"):
        return acc
    if epi == "relu":
        return relu(acc)
    if epi == "gate":
        return relu_grad(acc, gate)
    raise ValueError(epi)


# ---- convolutions --------------------------------------------------------
def conv2d_fwd(x, w, stride=1, pad=0, epi=None, gate=None):
    """y = epi(cross-correlation of x (NHWC) with w (KRSC)), fp64."""
    n, h, wd, c = x.shape
    k, r, s, c2 = w.shape
    assert c == c2
    sv = _shape_vec(n, h, wd, c, k, r, s, stride, pad)
    return _epilogue(_run_full(sv, OP_FWD, x, w), epi, gate)


def conv2d_bwd_data(dy, w, x_shape, stride=1, pad=0, epi=None, gate=None):
    """dx = epi(adjoint of conv2d_fwd w.r.t. x applied to dy), fp64."""
    n, h, wd, c = x_shape
    k, r, s, c2 = w.shape
    assert c == c2
    sv = _shape_vec(n, h, wd, c, k, r, s, stride, pad)
    assert out_dims(sv, OP_FWD) == tuple(dy.shape)
    return _epilogue(_run_full(sv, OP_BWD_DATA, dy, w), epi, gate)


def conv2d_bwd_weight(x, dy, r, s, stride=1, pad=0):
    """dW[k,r,s,c] = sum over n,p,q of dy * shifted x, fp64 (KRSC)."""
    n, h, wd, c = x.shape
    k = dy.shape[3]
    sv = _shape_vec(n, h, wd, c, k, r, s, stride, pad)
    assert out_dims(sv, OP_FWD) == tuple(dy.shape)
    return _run_full(sv, OP_BWD_WEIGHT, x, dy)


def conv_transpose2d_fwd(x, wt, stride=2, pad=1, epi=None, gate=None):
    """y = epi(transposed convolution of x (NHWC) with wt (C_in,R,S,C_out))."""
    n, h, wd, c = x.shape
    c2, r, s, k = wt.shape
    assert c == c2
    sv = _shape_vec(n, h, wd, c, k, r, s, stride, pad)
    return _epilogue(_run_full(sv, OP_CONVT, x, wt), epi, gate)


# ---- sampled versions: values at flat output indices ---------------------
def conv2d_fwd_points(x, w, idx, stride=1, pad=0):
    n, h, wd, c = x.shape
    k, r, s, _ = w.shape
    return _run_points(_shape_vec(n, h, wd, c, k, r, s, stride, pad), OP_FWD,
                       x, w, idx)


def conv2d_bwd_data_points(dy, w, x_shape, idx, stride=1, pad=0):
    n, h, wd, c = x_shape
    k, r, s, _ = w.shape
    return _run_points(_shape_vec(n, h, wd, c, k, r, s, stride, pad),
                       OP_BWD_DATA, dy, w, idx)


def conv2d_bwd_weight_points(x, dy, r, s, idx, stride=1, pad=0):
    n, h, wd, c = x.shape
    k = dy.shape[3]
    return _run_points(_shape_vec(n, h, wd, c, k, r, s, stride, pad),
                       OP_BWD_WEIGHT, x, dy, idx)


def conv_transpose2d_fwd_points(x, wt, idx, stride=2, pad=1):
    n, h, wd, c = x.shape
    _, r, s, k = wt.shape
    return _run_points(_shape_vec(n, h, wd, c, k, r, s, stride, pad),
                       OP_CONVT, x, wt, idx)


def conv_flops(n, p, q, k, c, r, s):
    """Direct-convolution operation count 2*N*P*Q*K*C*R*S (Section 5.2)."""
    return 2 * n * p * q * k * c * r * s
