"""GPU parity of the FC-DenseNet glue (Section 6.2): the Huber head
gradient, 2x2 average pooling and its gated gradient, and channel slice
copies (dense concatenation and its slice gradients). Each computes a
plainly defined value exactly and rounds it once, so the bar is bit
equality with the oracle, on ragged shapes (pixel counts that fill no
workgroup, channel counts that are multiples of 8 but not of 64, strides
above the copied width, channel offsets), with gates holding zeros, -0 and
negatives, and with overflow to infinity."""
import numpy as np
import pytest
import torch

import paper_1909_11150_amd as fg
from gpu_util import dev, host
from oracle import dense as D

pytestmark = pytest.mark.gpu


def _eq(a, b, what):
    a = np.asarray(a).view(np.uint16)
    b = np.asarray(b).view(np.uint16)
    bad = np.nonzero(a.ravel() != b.ravel())[0]
    assert bad.size == 0, f"{what}: {bad.size} differ, first at {bad[:5]}"


def _h(rng, shape, scale=1.0):
    return (rng.normal(size=shape) * scale).astype(np.float16)


@pytest.mark.parametrize("numel", [1, 7, 4099, 1 << 18])
@pytest.mark.parametrize("delta", [10.0, 0.5, np.inf])
def test_huber_head_grad(numel, delta):
    rng = np.random.default_rng(numel)
    y = _h(rng, numel, 12.0)
    t = (rng.normal(size=numel) * 12.0).astype(np.float32)
    S = 2.0 ** 13
    dy = torch.empty(numel, dtype=torch.float16, device="cuda")
    fg.huber_head_grad(dev(y), dev(t), S / numel, delta, dy)
    _eq(host(dy), D.huber_head_grad(y, t, S / numel, delta), "huber")


def test_huber_head_grad_overflow():
    y = np.array([1000.0, -1000.0, 1.0, -2.0, 0.0, 5.0, 7.0, 9.0], np.float16)
    t = np.zeros(8, np.float32)
    dy = torch.empty(8, dtype=torch.float16, device="cuda")
    fg.huber_head_grad(dev(y), dev(t), 2.0 ** 20, 100.0, dy)
    want = D.huber_head_grad(y, t, 2.0 ** 20, 100.0)
    assert want[0] == np.inf and want[1] == -np.inf
    _eq(host(dy), want, "huber overflow")


POOL = [(1, 2, 2, 8), (2, 6, 10, 24), (3, 34, 18, 72), (4, 128, 128, 256)]


@pytest.mark.parametrize("shape", POOL, ids=[str(s) for s in POOL])
def test_avg_pool2d(shape):
    n, h, w, c = shape
    rng = np.random.default_rng(h * w + c)
    x = _h(rng, shape, 3.0)
    y = torch.empty((n, h // 2, w // 2, c), dtype=torch.float16, device="cuda")
    fg.avg_pool2d_fwd(dev(x), y)
    _eq(host(y), D.avg_pool2d_fwd(x), "pool fwd")
    dy = _h(rng, (n, h // 2, w // 2, c), 1e-3)
    dy.ravel()[:8] = np.float16(6e-8)        # subnormals: a quarter rounds
    gate = _h(rng, shape)
    gate.ravel()[:16] = 0.0
    gate.ravel()[16:24] = np.float16(-0.0)
    for gt in (None, gate):
        dx = torch.empty(shape, dtype=torch.float16, device="cuda")
        fg.avg_pool2d_bwd(dev(dy), dx, None if gt is None else dev(gt))
        _eq(host(dx), D.avg_pool2d_bwd(dy, gt), f"pool bwd gate={gt is not None}")


@pytest.mark.parametrize("npix,nch,src_ld,dst_ld,off", [
    (1, 8, 8, 8, 0), (37, 24, 40, 64, 16), (4099, 256, 256, 1024, 768),
    (65536, 512, 768, 1280, 256)])
@pytest.mark.parametrize("gated,acc", [(False, False), (True, False), (True, True),
                                       (False, True)])
def test_channel_slice_copy(npix, nch, src_ld, dst_ld, off, gated, acc):
    rng = np.random.default_rng(npix + nch + off)
    src = _h(rng, (npix, src_ld))
    dst = _h(rng, (npix, dst_ld))
    gate = _h(rng, (npix, nch)) if gated else None
    if gated:
        gate.ravel()[:8] = 0.0
    if acc:
        dst[0, off:off + nch] = np.float16(60000.0)
        src[0, :nch] = np.float16(60000.0)
    ds, dd = dev(src), dev(dst)
    dg = dev(gate) if gated else None
    soff = 8 if src_ld >= nch + 8 else 0
    fg.channel_slice_copy(ds.data_ptr() + 2 * soff, src_ld, dd.data_ptr() + 2 * off, dst_ld,
                          npix, nch, gate=dg, gate_ld=nch if gated else 0, accumulate=acc)
    want = dst.copy()
    want[:, off:off + nch] = D.channel_slice_copy(src[:, soff:soff + nch],
                                                  dst[:, off:off + nch], gate, acc)
    _eq(host(dd), want, "slice copy")   # untouched channels stay as they were


def test_concat_then_slices_round_trip():
    """A dense block's concatenation written piece by piece into its channel
    slices, then each slice read back."""
    rng = np.random.default_rng(11)
    npix, widths = 3 * 17 * 9, (64, 256, 256, 256)
    pieces = [_h(rng, (npix, c)) for c in widths]
    total = sum(widths)
    z = torch.zeros((npix, total), dtype=torch.float16, device="cuda")
    off = 0
    for p in pieces:
        fg.channel_slice_copy(dev(p), p.shape[1], z.data_ptr() + 2 * off, total, npix,
                              p.shape[1])
        off += p.shape[1]
    _eq(host(z), D.concat_channels(pieces), "concat")
    off = 0
    for p in pieces:
        out = torch.empty_like(dev(p))
        fg.channel_slice_copy(z.data_ptr() + 2 * off, total, out, p.shape[1], npix,
                              p.shape[1])
        _eq(host(out), p, "slice")
        off += p.shape[1]
