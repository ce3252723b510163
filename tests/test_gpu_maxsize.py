"""GPU parity at the largest sizes the library accepts: every tensor holds
fewer than 2^31 elements (4 GiB of fp16), which takes each index
computation to its widest value.

  * Gradient path: one group of 2^31 - 4096 elements from two members (the
    second starting 2 GiB in), an infinity planted in its last element;
    pack, unscale with the check and unpack, compared bit for bit with the
    oracle on sampled elements and the group's ends, and the flag raised.
  * Convolution: a 3x3 layer whose input holds 2.13e9 elements (4.3 GB,
    beyond what a buffer resource addresses, so every pass takes the
    register-staged kernels), forward with ReLU, gated input gradient and
    kernel gradient on sampled outputs against the oracle.

Inputs are drawn on the device from seeded generators (2^31 host draws
would dominate the run time) and copied back for the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1909_11150_amd as fg
import synth
from gpu_util import conv_parity, host
from oracle import grad as G
from paper_1909_11150_amd import fcn

pytestmark = pytest.mark.gpu


def _sample(total, n, rng):
    idx = rng.integers(0, total, size=n, dtype=np.int64)
    ends = np.array([0, 1, 2, total - 3, total - 2, total - 1], np.int64)
    return np.unique(np.concatenate([idx, ends]))


def _take(t, idx):
    return t[torch.from_numpy(idx).to(t.device)].cpu().numpy()


def _patterns(n, gen):
    """fp16 bit patterns (as int16): finite values of every exponent and
    both signs."""
    v = torch.randint(0, 0x7C00, (n,), dtype=torch.int32, device="cuda", generator=gen)
    s = torch.randint(0, 2, (n,), dtype=torch.int32, device="cuda", generator=gen)
    return (v - 32768 * s).to(torch.int16)


def test_gradient_path_at_maximum_size():
    total = (1 << 31) - 4096
    n0 = 1 << 30
    numels = [n0, total - n0]
    plan = G.plan_groups(numels, 1 << 40, 256)
    assert len(plan) == 1 and plan[0]["numel"] == total
    grp = plan[0]
    gen = torch.Generator(device="cuda").manual_seed(11)
    srcs = [_patterns(n, gen) for n in numels]
    srcs[1][-1] = 0x7C00                      # +inf in the group's last element
    gbuf = torch.empty(total, dtype=torch.int16, device="cuda")
    fg.grad_group_pack([srcs[m] for m in grp["members"]], grp["offsets"], gbuf)
    g32 = torch.empty(total, dtype=torch.float32, device="cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    inv = np.float32(2.0 ** -15)
    fg.grad_unscale_check(gbuf, inv, g32, flag)
    dsts = [torch.empty(n, dtype=torch.float32, device="cuda") for n in numels]
    fg.grad_group_unpack(g32, [dsts[m] for m in grp["members"]], grp["offsets"])
    torch.cuda.synchronize()
    assert int(host(flag)[0]) == 1
    rng = np.random.default_rng(12)
    idx = _sample(total, 200_000, rng)
    off1 = grp["offsets"][grp["members"].index(1)]
    assert off1 == n0
    # the group holds member 0 then member 1, bit for bit
    got16 = _take(gbuf, idx).view(np.uint16)
    src16 = np.empty_like(got16)
    m0 = idx < n0
    src16[m0] = _take(srcs[0], idx[m0]).view(np.uint16)
    src16[~m0] = _take(srcs[1], idx[~m0] - n0).view(np.uint16)
    np.testing.assert_array_equal(got16, src16)
    # unscale: the oracle's single rounding of each sampled word
    r32 = G.unscale(src16, inv)
    np.testing.assert_array_equal(_take(g32, idx).view(np.uint32), r32.view(np.uint32))
    assert G.found_nonfinite(src16) == (total - 1 in set(idx.tolist()))
    # unpack: each member reads its own range of the fp32 group
    got0 = _take(dsts[0], idx[m0])
    got1 = _take(dsts[1], idx[~m0] - n0)
    np.testing.assert_array_equal(got0.view(np.uint32), r32[m0].view(np.uint32))
    np.testing.assert_array_equal(got1.view(np.uint32), r32[~m0].view(np.uint32))
    assert np.isinf(got1[-1]) and idx[-1] == total - 1


def test_conv_at_maximum_size():
    L = synth.Layer("MAX", "conv", (1, 2048, 1024, 1016), (1, 2048, 1024, 16), 3, 3, 1, 1,
                    True)
    assert int(np.prod(L.x_shape)) < (1 << 31) <= 2 * int(np.prod(L.x_shape))
    gen = torch.Generator(device="cuda").manual_seed(13)
    x = torch.randn(L.x_shape, dtype=torch.float16, device="cuda", generator=gen)
    x.relu_()
    w = (torch.randn(L.w_shape, dtype=torch.float32, device="cuda", generator=gen) *
         synth.he_std(L)).half()
    dy = torch.randn(L.y_shape, dtype=torch.float16, device="cuda", generator=gen)
    d = fcn.fwd_desc(L)
    for op in (fg.OP_FWD, fg.OP_BWD_DATA, fg.OP_BWD_WEIGHT):
        name = fg.kernel_name(d, op)
        print(op, name)
        assert "dma" not in name and "halo" not in name, name
    ws = torch.empty(max(16, fcn.chain_workspace_bytes([L])), dtype=torch.uint8,
                     device="cuda")
    y = torch.empty(L.y_shape, dtype=torch.float16, device="cuda")
    dx = torch.empty(L.x_shape, dtype=torch.float16, device="cuda")
    dw = torch.empty(L.w_shape, dtype=torch.float16, device="cuda")
    fg.conv2d_fwd(d, x, w, y, fg.EPI_RELU, None, ws)
    fg.conv2d_bwd_data(d, dy, w, dx, fg.EPI_GATE, x, ws)
    fg.conv2d_bwd_weight(d, x, dy, dw, ws)
    torch.cuda.synchronize()
    xh, wh, dyh = host(x), host(w), host(dy)
    rng = np.random.default_rng(14)
    iy = _sample(int(np.prod(L.y_shape)), 2000, rng)
    ref = oracle.relu(oracle.conv2d_fwd_points(xh, wh, iy, 1, 1))
    conv_parity(_take(y.view(-1), iy), ref, "fwd")
    ix = _sample(int(np.prod(L.x_shape)), 2000, rng)
    ref = oracle.conv2d_bwd_data_points(dyh, wh, xh.shape, ix, 1, 1)
    ref = np.where(xh.ravel()[ix].astype(np.float64) > 0, ref, 0.0)
    conv_parity(_take(dx.view(-1), ix), ref, "dx")
    iw = _sample(int(np.prod(L.w_shape)), 200, rng)
    ref = oracle.conv2d_bwd_weight_points(xh, dyh, 3, 3, iw, 1, 1)
    conv_parity(host(dw).ravel()[iw], ref, "dW")
