"""Pins for the fp64 convolution oracle (CPU only).

Nothing here compares the oracle with itself. Each test checks it against
something fixed independently of its source:
  * PyTorch's float64 CPU convolution and its autograd (a library routine),
  * an operator materialised column by column, against an im2col product
    written with padding and strided slicing,
  * closed forms (identity and delta kernels, all-ones tap counts),
  * exact identities of the mathematics (adjointness; central differences
    of a linear map are exact),
  * and the fp16 rounding of a closed-form value that lands on a tie.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth

CASES = [
    # n, h, w, c, k, r, s, stride, pad
    (1, 5, 5, 2, 3, 3, 3, 1, 1),
    (2, 6, 7, 3, 2, 3, 3, 2, 1),
    (1, 7, 6, 2, 2, 3, 2, 2, 0),
    (2, 4, 4, 4, 5, 1, 1, 1, 0),
    (1, 8, 8, 3, 2, 4, 4, 2, 1),
    (1, 9, 5, 2, 3, 3, 3, 3, 2),
]


def _rand(rng, shape):
    return synth.to_f16(rng.uniform(-1, 1, size=shape))


def _nchw(a):
    return torch.from_numpy(np.ascontiguousarray(
        np.asarray(a, np.float64).transpose(0, 3, 1, 2)))


def _kcrs(w):
    return torch.from_numpy(np.ascontiguousarray(
        np.asarray(w, np.float64).transpose(0, 3, 1, 2)))


def _nhwc(t):
    return t.detach().numpy().transpose(0, 2, 3, 1)


@pytest.mark.parametrize("case", CASES)
def test_fwd_bwd_match_torch_float64(oracle_lib, case):
    o = oracle_lib
    n, h, w, c, k, r, s, st, pd = case
    rng = np.random.default_rng(11)
    x = _rand(rng, (n, h, w, c))
    W = _rand(rng, (k, r, s, c))
    xt = _nchw(x).requires_grad_(True)
    Wt = _kcrs(W).requires_grad_(True)
    yt = F.conv2d(xt, Wt, stride=st, padding=pd)
    y = o.conv2d_fwd(x, W, st, pd)
    np.testing.assert_allclose(y, _nhwc(yt), rtol=1e-12, atol=1e-12)

    dy = _rand(rng, y.shape)
    yt.backward(_nchw(dy))
    dx = o.conv2d_bwd_data(dy, W, x.shape, st, pd)
    dW = o.conv2d_bwd_weight(x, dy, r, s, st, pd)
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW, Wt.grad.numpy().transpose(0, 2, 3, 1),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", [(1, 4, 4, 3, 2), (2, 5, 3, 2, 4), (1, 1, 1, 2, 3)])
def test_convt_matches_torch_float64(oracle_lib, case):
    o = oracle_lib
    n, h, w, ci, co = case
    rng = np.random.default_rng(12)
    x = _rand(rng, (n, h, w, ci))
    Wt = _rand(rng, (ci, 4, 4, co))
    xt = _nchw(x).requires_grad_(True)
    wt = torch.from_numpy(np.ascontiguousarray(
        Wt.astype(np.float64).transpose(0, 3, 1, 2))).requires_grad_(True)
    yt = F.conv_transpose2d(xt, wt, stride=2, padding=1)
    y = o.conv_transpose2d_fwd(x, Wt, 2, 1)
    assert y.shape == (n, 2 * h, 2 * w, co)
    np.testing.assert_allclose(y, _nhwc(yt), rtol=1e-12, atol=1e-12)
    # its backward passes, as the network's chain forms them
    from oracle import chain
    from synth import Layer
    L = Layer("t", "convT", x.shape, y.shape, 4, 4, 2, 1, False)
    dy = _rand(rng, y.shape)
    yt.backward(_nchw(dy))
    dx, dw = chain.layer_backward(L, x, Wt, dy, gate_input=False)
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy().transpose(0, 2, 3, 1),
                               rtol=1e-12, atol=1e-12)


def _im2col_fwd(x, W, st, pd):
    """Independent forward: zero-pad, slice strided windows, one matmul."""
    n, h, w, c = x.shape
    k, r, s, _ = W.shape
    xp = np.pad(x.astype(np.float64), ((0, 0), (pd, pd), (pd, pd), (0, 0)))
    P = (h + 2 * pd - r) // st + 1
    Q = (w + 2 * pd - s) // st + 1
    cols = np.stack([xp[:, i:i + st * (P - 1) + 1:st, j:j + st * (Q - 1) + 1:st, :]
                     for i in range(r) for j in range(s)], axis=3)
    cols = cols.reshape(n * P * Q, r * s * c)
    return (cols @ W.astype(np.float64).reshape(k, -1).T).reshape(n, P, Q, k)


@pytest.mark.parametrize("case", CASES[:4])
def test_materialised_operator(oracle_lib, case):
    """Build A column by column from unit inputs; check fwd = A, bwd_data = A^T."""
    o = oracle_lib
    n, h, w, c, k, r, s, st, pd = case
    rng = np.random.default_rng(13)
    W = _rand(rng, (k, r, s, c))
    nin = n * h * w * c
    cols = []
    for j in range(nin):
        e = np.zeros(nin)
        e[j] = 1.0
        cols.append(o.conv2d_fwd(e.reshape(n, h, w, c), W, st, pd).ravel())
    A = np.stack(cols, axis=1)
    x = _rand(rng, (n, h, w, c))
    np.testing.assert_allclose(A @ x.astype(np.float64).ravel(),
                               _im2col_fwd(x, W, st, pd).ravel(), atol=1e-12)
    y_shape = o.conv2d_fwd(x, W, st, pd).shape
    dy = _rand(rng, y_shape)
    np.testing.assert_allclose(o.conv2d_bwd_data(dy, W, x.shape, st, pd).ravel(),
                               A.T @ dy.astype(np.float64).ravel(), atol=1e-12)


def test_closed_forms_fwd(oracle_lib):
    o = oracle_lib
    rng = np.random.default_rng(14)
    x = _rand(rng, (2, 6, 5, 4))
    # 1x1 identity weight
    eye = np.eye(4, dtype=np.float16).reshape(4, 1, 1, 4)
    np.testing.assert_array_equal(o.conv2d_fwd(x, eye, 1, 0), x.astype(np.float64))
    # 3x3 centre delta, s1 p1
    d = np.zeros((4, 3, 3, 4), np.float16)
    for i in range(4):
        d[i, 1, 1, i] = 1
    np.testing.assert_array_equal(o.conv2d_fwd(x, d, 1, 1), x.astype(np.float64))
    # off-centre delta at (0, 2): y[p, q] = x[p-1, q+1], zero outside
    d2 = np.zeros((4, 3, 3, 4), np.float16)
    for i in range(4):
        d2[i, 0, 2, i] = 1
    y = o.conv2d_fwd(x, d2, 1, 1)
    ref = np.zeros_like(y)
    ref[:, 1:, :-1, :] = x[:, :-1, 1:, :]
    np.testing.assert_array_equal(y, ref)
    # 3x3 s2 p1 centre delta is a stride-2 subsample
    np.testing.assert_array_equal(o.conv2d_fwd(x, d, 2, 1),
                                  x[:, ::2, ::2, :].astype(np.float64))
    # all ones: C * (number of in-image taps): 4 corner / 6 edge / 9 interior
    ones = np.ones((1, 5, 5, 2), np.float16)
    y = o.conv2d_fwd(ones, np.ones((1, 3, 3, 2), np.float16), 1, 1)[0, :, :, 0]
    assert y[0, 0] == 8 and y[0, 2] == 12 and y[2, 2] == 18 and y[4, 4] == 8


def test_bwd_data_tap_counts_stride2(oracle_lib):
    """3x3 s2 p1 all-ones: taps per row are 1 for even h, 2 for odd h, and 1
    for the last odd row (its lower neighbour is outside the output)."""
    o = oracle_lib
    x_shape = (1, 8, 8, 1)
    dy = np.ones((1, 4, 4, 1), np.float16)
    dx = o.conv2d_bwd_data(dy, np.ones((1, 3, 3, 1), np.float16), x_shape, 2, 1)
    t = np.array([1, 2, 1, 2, 1, 2, 1, 1], dtype=np.float64)
    np.testing.assert_array_equal(dx[0, :, :, 0], np.outer(t, t))


def test_adjoint_identity(oracle_lib):
    o = oracle_lib
    rng = np.random.default_rng(15)
    for (n, h, w, c, k, r, s, st, pd) in CASES:
        x = _rand(rng, (n, h, w, c))
        W = _rand(rng, (k, r, s, c))
        y = o.conv2d_fwd(x, W, st, pd)
        dy = _rand(rng, y.shape)
        lhs = float(np.sum(y * dy.astype(np.float64)))
        rhs = float(np.sum(x.astype(np.float64) *
                           o.conv2d_bwd_data(dy, W, x.shape, st, pd)))
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


def test_bwd_weight_central_differences(oracle_lib):
    """f(W) = <fwd(x; W), dy> is linear in W, so a central difference with
    step 1 is exact and equals dW elementwise."""
    o = oracle_lib
    rng = np.random.default_rng(16)
    n, h, w, c, k, r, s, st, pd = (1, 5, 6, 2, 2, 3, 3, 2, 1)
    x = _rand(rng, (n, h, w, c))
    W = _rand(rng, (k, r, s, c)).astype(np.float64)
    dy = _rand(rng, o.conv2d_fwd(x, W, st, pd).shape).astype(np.float64)
    dW = o.conv2d_bwd_weight(x, dy, r, s, st, pd)

    def f(Wv):
        return float(np.sum(o.conv2d_fwd(x, Wv, st, pd) * dy))

    fd = np.zeros_like(W)
    for idx in np.ndindex(W.shape):
        e = np.zeros_like(W)
        e[idx] = 1.0
        fd[idx] = (f(W + e) - f(W - e)) / 2.0
    np.testing.assert_allclose(dW, fd, rtol=1e-12, atol=1e-12)


def test_bwd_weight_all_ones_closed_form(oracle_lib):
    """x = dy = 1: dW[k,r,s,c] = N * cnt_h(r) * cnt_w(s).

    Single 3x3 s1 p1 conv at 64x64, N=2: counts (63, 64, 63) give
    7938, 8064, 8192; fp16 nearest-even turns the 7938 tie into 7936."""
    o = oracle_lib
    x = np.ones((2, 64, 64, 16), np.float16)
    dy = np.ones((2, 64, 64, 16), np.float16)
    dW = o.conv2d_bwd_weight(x, dy, 3, 3, 1, 1)
    assert dW.shape == (16, 3, 3, 16)
    cnt = np.array([63, 64, 63])
    np.testing.assert_array_equal(dW[0, :, :, 0], 2 * np.outer(cnt, cnt))
    assert dW[5, 0, 0, 7] == 7938
    h = dW.astype(np.float16)
    assert h[0, 0, 0, 0] == 7936 and h[0, 0, 1, 0] == 8064 and h[0, 1, 1, 0] == 8192
    # 3x3 s2 p1 at 128: counts (63, 64, 64)
    x2 = np.ones((1, 128, 128, 1), np.float16)
    dy2 = np.ones((1, 64, 64, 1), np.float16)
    dW2 = o.conv2d_bwd_weight(x2, dy2, 3, 3, 2, 1)
    cnt2 = np.array([63, 64, 64])
    np.testing.assert_array_equal(dW2[0, :, :, 0], np.outer(cnt2, cnt2))


def test_convt_closed_forms(oracle_lib):
    o = oracle_lib
    rng = np.random.default_rng(17)
    x = _rand(rng, (1, 4, 5, 3))
    # delta at tap (1,1): zero-insertion upsampling y[2i, 2j] = x[i, j]
    Wt = np.zeros((3, 4, 4, 3), np.float16)
    for i in range(3):
        Wt[i, 1, 1, i] = 1
    y = o.conv_transpose2d_fwd(x, Wt, 2, 1)
    ref = np.zeros((1, 8, 10, 3))
    ref[:, ::2, ::2, :] = x
    np.testing.assert_array_equal(y, ref)
    # all ones: C_in * t(o) * t(u), t = 1 on the first/last row, 2 inside
    y1 = o.conv_transpose2d_fwd(np.ones((1, 4, 4, 3), np.float16),
                                np.ones((3, 4, 4, 1), np.float16), 2, 1)
    t = np.array([1, 2, 2, 2, 2, 2, 2, 1], dtype=np.float64)
    np.testing.assert_array_equal(y1[0, :, :, 0], 3 * np.outer(t, t))


def test_convt_equals_bwd_data_with_roles_exchanged(oracle_lib):
    """convT(x; Wt) is the input gradient of the conv whose KRSC weight is
    Wt (K = C_in, C = C_out): the same value, evaluated by another formula."""
    o = oracle_lib
    rng = np.random.default_rng(18)
    x = _rand(rng, (2, 5, 4, 3))
    Wt = _rand(rng, (3, 4, 4, 2))
    y = o.conv_transpose2d_fwd(x, Wt, 2, 1)
    dx = o.conv2d_bwd_data(x, Wt, (2, 10, 8, 2), 2, 1)
    np.testing.assert_allclose(y, dx, rtol=1e-14, atol=1e-14)


def test_epilogues():
    import oracle
    acc = np.array([1.5, -2.0, 0.0, -0.0, 3.0])
    r = oracle.relu(acc)
    np.testing.assert_array_equal(r, [1.5, 0, 0, 0, 3.0])
    assert not np.signbit(r[1]) and not np.signbit(r[3])
    gate = np.array([1.0, 2.0, 0.0, 1.0, -1.0], np.float16)
    g = oracle.relu_grad(acc, gate)
    np.testing.assert_array_equal(g, [1.5, -2.0, 0.0, -0.0, 0.0])
    assert not np.signbit(g[4])


def test_points_agree_with_definition_by_index(oracle_lib):
    """Sampled evaluation returns the value at each flat index of the full
    output for every operation (index decoding and op selection)."""
    o = oracle_lib
    rng = np.random.default_rng(19)
    n, h, w, c, k, r, s, st, pd = (2, 6, 7, 3, 4, 3, 3, 2, 1)
    x = _rand(rng, (n, h, w, c))
    W = _rand(rng, (k, r, s, c))
    y = o.conv2d_fwd(x, W, st, pd)
    dy = _rand(rng, y.shape)
    Wt = _rand(rng, (c, 4, 4, k))
    full = {
        "fwd": (y, lambda i: o.conv2d_fwd_points(x, W, i, st, pd)),
        "bwd_data": (o.conv2d_bwd_data(dy, W, x.shape, st, pd),
                     lambda i: o.conv2d_bwd_data_points(dy, W, x.shape, i, st, pd)),
        "bwd_weight": (o.conv2d_bwd_weight(x, dy, r, s, st, pd),
                       lambda i: o.conv2d_bwd_weight_points(x, dy, r, s, i, st, pd)),
        "convt": (o.conv_transpose2d_fwd(x, Wt, 2, 1),
                  lambda i: o.conv_transpose2d_fwd_points(x, Wt, i, 2, 1)),
    }
    for name, (ref, fn) in full.items():
        idx = rng.choice(ref.size, size=min(50, ref.size), replace=False)
        np.testing.assert_array_equal(fn(idx), ref.ravel()[idx], err_msg=name)
