"""The kernel gradient without a workspace argument
(conv2d_bwd_weight_noalloc, for callers that cannot allocate) against
conv2d_bwd_weight with a caller workspace, both called through the C ABI:
bit for bit where the regular call's workspace fits the library's static
scratch (same plan, same kernels), and to the single-op rule where the
scratch limits the split count. Calls run back to back on one stream, a
smaller input after a larger one, so each reads scratch the previous call
left behind."""
import ctypes

import numpy as np
import pytest
import torch

import paper_1909_11150_amd as fg
import synth
from gpu_util import conv_parity, dev, empty16, host, workspace

pytestmark = pytest.mark.gpu


def _inputs(shape, seed):
    n, h, w, c, k, r, st, pd = shape
    rng = np.random.default_rng(seed)
    d = fg.ConvDesc.make(n, h, w, c, k, r, r, st, pd)
    p, q = fg.out_dims(d)
    x = np.maximum(synth.normal(rng, (n, h, w, c)), np.float16(0))
    dy = synth.normal(rng, (n, p, q, k))
    return d, dev(x), dev(dy), (k, r, r, c)


def _noalloc(d, x, dy, dw):
    st = fg.lib().conv2d_bwd_weight_noalloc(ctypes.byref(d), x.data_ptr(), dy.data_ptr(),
                                            dw.data_ptr(),
                                            torch.cuda.current_stream().cuda_stream)
    assert st == fg.FG_OK, fg.status_string(st)


def _regular(d, x, dy, dw, ws):
    st = fg.lib().conv2d_bwd_weight(ctypes.byref(d), x.data_ptr(), dy.data_ptr(),
                                    dw.data_ptr(), ws.data_ptr(), ws.numel(),
                                    torch.cuda.current_stream().cuda_stream)
    assert st == fg.FG_OK, fg.status_string(st)


def test_two_calls_in_a_row_match_the_workspace_call():
    shapes = [(4, 128, 128, 512, 512, 3, 1, 1),   # 63 MiB of split partials
              (1, 77, 79, 512, 512, 3, 1, 1)]     # smaller, fewer partials
    runs = [_inputs(s, 40 + i) for i, s in enumerate(shapes)]
    for d, *_ in runs:
        need = fg.workspace_bytes(d, fg.OP_BWD_WEIGHT)
        assert 0 < need <= fg.NOALLOC_SCRATCH_BYTES
    outs = []
    for d, x, dy, wsh in runs:            # the two no-allocation calls in a row
        dw = empty16(wsh)
        _noalloc(d, x, dy, dw)
        outs.append(dw)
    for (d, x, dy, wsh), got in zip(runs, outs):
        ref = empty16(wsh)
        _regular(d, x, dy, ref, workspace(d, fg.OP_BWD_WEIGHT))
        np.testing.assert_array_equal(host(got).view(np.uint16), host(ref).view(np.uint16))


def test_plan_limited_by_the_scratch_and_the_head():
    """A shape whose best plan needs more than the scratch (fewer splits:
    same sum, another fp32 order) and the 1x1 head's kernel gradient, again
    twice in a row, the second smaller."""
    shapes = [(4, 64, 64, 1024, 1024, 3, 1, 1), (2, 30, 30, 64, 1, 1, 1, 0)]
    runs = [_inputs(s, 50 + i) for i, s in enumerate(shapes)]
    assert fg.workspace_bytes(runs[0][0], fg.OP_BWD_WEIGHT) > fg.NOALLOC_SCRATCH_BYTES
    outs = []
    for d, x, dy, wsh in runs:
        dw = empty16(wsh)
        _noalloc(d, x, dy, dw)
        outs.append(dw)
    for i, ((d, x, dy, wsh), got) in enumerate(zip(runs, outs)):
        ref = empty16(wsh)
        _regular(d, x, dy, ref, workspace(d, fg.OP_BWD_WEIGHT))
        if i == 0:
            conv_parity(host(got), host(ref).astype(np.float64), "capped plan")
        else:
            np.testing.assert_array_equal(host(got).view(np.uint16),
                                          host(ref).view(np.uint16))
