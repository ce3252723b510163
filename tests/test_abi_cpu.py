"""C-ABI checks that need no GPU: the library loads, exports every function
the header declares, validates arguments on the host (no device call is made
on these paths) and plans the gradient groups."""
import ctypes
import json
import os
import re

import numpy as np
import pytest

import paper_1909_11150_amd as fg
import synth
from oracle import grad as G

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fcngrad.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(fg.LIB_PATH):
        from paper_1909_11150_amd import build
        build.build()
    return fg.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(",
                                 text, flags=re.M)))


def test_header_declares_the_seven_passes_and_helpers():
    names = declared_functions()
    for n in ("conv2d_fwd", "conv2d_bwd_data", "conv2d_bwd_weight",
              "conv_transpose2d_fwd", "grad_group_pack", "grad_unscale_check",
              "grad_group_unpack"):
        assert n in names
    assert set(names) == set(fg.ENTRY_POINTS)


def test_library_exports_every_declared_symbol(L):
    for n in declared_functions():
        assert hasattr(L, n), n


def _desc(**kw):
    base = dict(n=2, h=8, w=8, c=16, k=16, r=3, s=3, stride=1, pad=1)
    base.update(kw)
    return fg.ConvDesc.make(**base)


FAKE = 0x1000  # never dereferenced: every call below fails validation


def test_invalid_arguments_return_einval(L):
    d = _desc()
    ref = ctypes.byref
    assert L.conv2d_fwd(None, FAKE, FAKE + 4096, FAKE + 8192, 0, None, None, 0, None) == fg.FG_EINVAL
    assert L.conv2d_fwd(ref(d), None, FAKE, FAKE + 8192, 0, None, None, 0, None) == fg.FG_EINVAL
    # gate required for the gate epilogue
    assert L.conv2d_fwd(ref(d), FAKE, FAKE + 1 << 20, FAKE + 1 << 22, fg.EPI_GATE,
                        None, None, 0, None) == fg.FG_EINVAL
    # unknown epilogue
    assert L.conv2d_fwd(ref(d), FAKE, FAKE + (1 << 20), FAKE + (1 << 22), 7,
                        None, None, 0, None) == fg.FG_EINVAL
    # output aliasing the input
    assert L.conv2d_fwd(ref(d), FAKE, FAKE + (1 << 20), FAKE, 0, None, None, 0,
                        None) == fg.FG_EINVAL
    # non-positive sizes and a kernel that does not fit
    for bad in (_desc(n=0), _desc(c=-8), _desc(r=11, pad=0), _desc(stride=0)):
        assert L.conv2d_fwd(ref(bad), FAKE, FAKE + (1 << 20), FAKE + (1 << 22), 0,
                            None, None, 0, None) == fg.FG_EINVAL
    # kernel gradient with the non-finite flag: the flag is required and
    # must not alias dW (x at FAKE, dy at +1 MiB, dW at +4 MiB)
    x, dy, dw = FAKE, FAKE + (1 << 20), FAKE + (1 << 22)
    assert L.conv2d_bwd_weight_checked(ref(d), x, dy, dw, None, None, 0,
                                       None) == fg.FG_EINVAL
    assert L.conv2d_bwd_weight_checked(ref(d), x, dy, dw, dw + 8, None, 0,
                                       None) == fg.FG_EINVAL
    assert L.conv2d_bwd_weight_checked(ref(d), x, dy, dw, x, None, 0,
                                       None) == fg.FG_EINVAL
    # gradient path
    seg = (fg.Segment * 1)(fg.Segment(FAKE, 10, 0))
    assert L.grad_group_pack(seg, 0, FAKE + 4096, 10, None) == fg.FG_EINVAL
    assert L.grad_group_pack(seg, 1, FAKE + 4096, 5, None) == fg.FG_EINVAL  # outside
    two = (fg.Segment * 2)(fg.Segment(FAKE, 10, 0), fg.Segment(FAKE + 64, 10, 5))
    assert L.grad_group_pack(two, 2, FAKE + 4096, 64, None) == fg.FG_EINVAL  # overlap
    assert L.grad_unscale_check(FAKE, 0, 1.0, FAKE + 4096, FAKE + 8192, None) == fg.FG_EINVAL
    assert L.grad_unscale_check(FAKE, 100, 1.0, FAKE + 100, FAKE + 8192, None) == fg.FG_EINVAL
    assert L.grad_group_unpack(FAKE, 10, seg, 1, None) == fg.FG_EINVAL  # dst overlaps group
    assert L.l2_head_grad(FAKE, FAKE + 4096, 10, 1.0, FAKE, None) == fg.FG_EINVAL
    assert L.relu_backward(None, FAKE, 10, FAKE + 4096, None) == fg.FG_EINVAL


def test_unsupported_shapes(L):
    ref = ctypes.byref
    for bad in (_desc(c=12), _desc(k=12), _desc(k=1, r=3), _desc(r=5, s=5, pad=2)):
        assert L.conv2d_fwd(ref(bad), FAKE, FAKE + (1 << 20), FAKE + (1 << 22), 0,
                            None, None, 0, None) == fg.FG_EUNSUPPORTED
    # transposed conv is implemented for 4x4 stride 2 pad 1 only
    t = fg.ConvDesc.make(1, 4, 4, 16, 16, 3, 3, 2, 1)
    assert L.conv_transpose2d_fwd(ref(t), FAKE, FAKE + (1 << 20), FAKE + (1 << 22),
                                  0, None, None, 0, None) == fg.FG_EUNSUPPORTED
    segs = (fg.Segment * 65)(*[fg.Segment(FAKE + 64 * i, 1, i) for i in range(65)])
    assert L.grad_group_pack(segs, 65, FAKE + (1 << 20), 65, None) == fg.FG_EUNSUPPORTED


def test_workspace_query_and_shortfall(L):
    ref = ctypes.byref
    d = fg.ConvDesc.make(4, 64, 64, 512, 1024, 3, 3, 2, 1)
    need = L.fg_conv_workspace_bytes(ref(d), fg.OP_BWD_WEIGHT)
    assert need > 0 and need % 4 == 0
    # a shape with few output tiles splits its reduction and needs workspace
    small = fg.ConvDesc.make(4, 32, 32, 1024, 1024, 3, 3, 2, 1)
    assert L.fg_conv_workspace_bytes(ref(small), fg.OP_FWD) > 0
    assert L.conv2d_fwd(ref(small), FAKE, FAKE + (1 << 28), FAKE + (1 << 30), 0, None,
                        None, 0, None) == fg.FG_EWORKSPACE
    # a large one does not
    big = fg.ConvDesc.make(4, 128, 128, 512, 512, 3, 3, 1, 1)
    assert L.fg_conv_workspace_bytes(ref(big), fg.OP_FWD) == 0
    assert L.conv2d_bwd_weight(ref(d), FAKE, FAKE + (1 << 28), FAKE + (1 << 30),
                               None, 0, None) == fg.FG_EWORKSPACE
    assert L.conv2d_bwd_weight(ref(d), FAKE, FAKE + (1 << 28), FAKE + (1 << 30),
                               FAKE + (1 << 32), need - 4, None) == fg.FG_EWORKSPACE
    head = fg.ConvDesc.make(4, 256, 256, 256, 1, 1, 1, 1, 0)
    assert L.fg_conv_workspace_bytes(ref(head), fg.OP_BWD_WEIGHT) > 0


def test_small_tile_plans_keep_one_workgroup_per_cu(L):
    """The 16x16 layers' passes on 128x128 tiles split their reduction only
    as far as one workgroup per CU (at most 256 workgroups): such a
    workgroup, alone on its CU, runs faster than two sharing one, so filling
    the second slot with more splits loses."""
    from paper_1909_11150_amd.fcn import convt_dx_desc, fwd_desc
    layers = {l.name: l for l in synth.fcn_layers()}
    cases = {  # pass: (descriptor, op, output shape, 128x128 tiles, expected splits)
        "E4a.fwd": (fwd_desc(layers["E4a"]), fg.OP_FWD, layers["E4a"].y_shape, 64, 4),
        "E4b.fwd": (fwd_desc(layers["E4b"]), fg.OP_FWD, layers["E4b"].y_shape, 64, 4),
        "E4b.dx": (fwd_desc(layers["E4b"]), fg.OP_BWD_DATA, layers["E4b"].x_shape, 64, 4),
        "E4a.dx": (fwd_desc(layers["E4a"]), fg.OP_BWD_DATA, layers["E4a"].x_shape, 256, 1),
        "D4T.fwd": (fwd_desc(layers["D4T"]), fg.OP_CONVT, layers["D4T"].y_shape, 256, 1),
    }
    for name, (d, op, shape, tiles, splits) in cases.items():
        kern = fg.kernel_name(d, op)
        assert kern.startswith("data_conv_dma_kernel<128,"), (name, kern)
        ws = L.fg_conv_workspace_bytes(ctypes.byref(d), op)
        got = ws // (4 * int(np.prod(shape))) if ws else 1
        assert got == splits and tiles * got <= 256, (name, got)
    # the transposed convolution's input gradient keeps 256x256 tiles
    assert fg.kernel_name(convt_dx_desc(layers["D4T"]), fg.OP_FWD).startswith(
        "data_conv_dma_kernel<true")


def test_kernel_gradients_without_big_tiles_split_widely(L):
    """A kernel gradient whose R*S*C or K is below 256 has only 128x128
    tiles, and few of them: it may split its reduction beyond 16 ways to
    fill the GPU; shapes with 256x256 tiles (the network's layers) keep 16
    at most."""
    def splits(d):
        ws = L.fg_conv_workspace_bytes(ctypes.byref(d), fg.OP_BWD_WEIGHT)
        return ws // (4 * d.k * d.r * d.s * d.c) if ws else 1
    one_by_one = fg.ConvDesc.make(8, 64, 64, 128, 64, 1, 1, 1, 0)  # one 128x128 tile
    assert fg.kernel_name(one_by_one, fg.OP_BWD_WEIGHT) == "wgrad_kernel<Cfg<128, 128, 2, 2>, true>"
    assert splits(one_by_one) > 16
    from paper_1909_11150_amd.fcn import convt_dx_desc, fwd_desc
    for l in synth.fcn_layers():
        d = fwd_desc(l) if l.kind == "conv" else convt_dx_desc(l)
        if d.k * d.r * d.s * d.c >= 256 * 256:
            assert splits(d) <= 16, l.name


def test_out_dims_match_layer_table():
    for L_ in synth.fcn_layers():
        n, h, w, c = L_.x_shape
        d = fg.ConvDesc.make(n, h, w, c, L_.y_shape[3], L_.r, L_.s, L_.stride, L_.pad)
        assert fg.out_dims(d, transpose=(L_.kind == "convT")) == L_.y_shape[1:3]


def test_library_planner_matches_golden_and_oracle():
    with open(os.path.join(ROOT, "tests", "golden", "fcn_groups.json")) as f:
        gold = json.load(f)
    gof, oof, gnum = fg.grad_group_plan(gold["numels"], gold["cap_bytes"],
                                        gold["align_bytes"], 2)
    assert gnum == [g["numel"] for g in gold["groups"]]
    names = gold["completion_order"]
    members = [[names[i] for i in range(len(names)) if gof[i] == g]
               for g in range(len(gnum))]
    assert members == [g["members"] for g in gold["groups"]]
    # small cases against the oracle planner
    import numpy as np
    rng = np.random.default_rng(3)
    for _ in range(50):
        numels = [int(v) for v in rng.integers(1, 3000, size=rng.integers(1, 12))]
        cap = int(rng.integers(512, 8192))
        plan = G.plan_groups(numels, cap, 256)
        gof, oof, gnum = fg.grad_group_plan(numels, cap, 256, 2)
        assert gnum == [p["numel"] for p in plan]
        for gi, p in enumerate(plan):
            for m, off in zip(p["members"], p["offsets"]):
                assert gof[m] == gi and oof[m] == off


def test_status_strings(L):
    assert fg.status_string(fg.FG_EWORKSPACE).startswith("FG_EWORKSPACE")


def test_optimizer_argument_checks(L):
    """lars_adam_update rejects bad layers, parameters and workspace before
    touching the device (no pointer below is dereferenced)."""
    ref = ctypes.byref
    n = 1024

    def layer(base):  # w32, w16, m, v, g laid out 64 KiB apart
        return fg.OptTensor(base, base + (1 << 16), base + (2 << 16), base + (3 << 16),
                            base + (4 << 16), n)

    good = (fg.OptTensor * 2)(layer(FAKE), layer(FAKE + (1 << 20)))
    p = fg.OptParams(1e-3, 0.9, 0.999, 1e-8, 1e-4)
    sc, ws = FAKE + (1 << 24), FAKE + (1 << 25)
    need = L.fg_lars_adam_workspace_bytes(good, 2)
    assert need > 0
    assert L.lars_adam_update(good, 0, ref(p), None, 0, sc, ws, need, None) == fg.FG_EINVAL
    assert L.lars_adam_update(good, 2, ref(p), None, 0, None, ws, need, None) == fg.FG_EINVAL
    assert L.lars_adam_update(good, 2, ref(p), None, 3, sc, ws, need, None) == fg.FG_EINVAL
    assert L.lars_adam_update(good, 2, ref(p), None, 0, sc, ws, need - 4, None) == fg.FG_EWORKSPACE
    for bad in (fg.OptParams(-1.0, 0.9, 0.999, 1e-8, 0.0), fg.OptParams(1e-3, 1.0, 0.999, 1e-8, 0.0),
                fg.OptParams(1e-3, 0.9, 0.999, -1.0, 0.0), fg.OptParams(float("nan"), 0.9, 0.999, 0.0, 0.0)):
        assert L.lars_adam_update(good, 2, ref(bad), None, 0, sc, ws, need, None) == fg.FG_EINVAL
    mis = (fg.OptTensor * 1)(fg.OptTensor(FAKE + 4, FAKE + (1 << 16), FAKE + (2 << 16),
                                          FAKE + (3 << 16), FAKE + (4 << 16), n))
    assert L.lars_adam_update(mis, 1, ref(p), None, 0, sc, ws, need, None) == fg.FG_EINVAL
    alias = (fg.OptTensor * 2)(layer(FAKE), layer(FAKE + 2048))  # second w32 inside the first
    assert L.lars_adam_update(alias, 2, ref(p), None, 0, sc, ws, need, None) == fg.FG_EINVAL
    assert L.lars_adam_update(good, 2, ref(p), None, 0, FAKE + 64, ws, need, None) == fg.FG_EINVAL
    # flags inside memory the update writes: the step count, the workspace, a weight
    for bad_flags in (sc, ws + 16, FAKE + 8):
        assert L.lars_adam_update(good, 2, ref(p), bad_flags, 2, sc, ws, need,
                                  None) == fg.FG_EINVAL


def test_optimizer_split_argument_checks(L):
    """lars_adam_norms / lars_adam_apply reject bad ranges, gradient forms
    and scales, and an apply without norms, before touching the device."""
    ref = ctypes.byref
    n = 1024

    def layer(base, g_off=4 << 16):
        return fg.OptTensor(base, base + (1 << 16), base + (2 << 16), base + (3 << 16),
                            base + g_off, n)

    good = (fg.OptTensor * 2)(layer(FAKE), layer(FAKE + (1 << 20)))
    p = fg.OptParams(1e-3, 0.9, 0.999, 1e-8, 1e-4)
    sc, ws = FAKE + (1 << 24), FAKE + (1 << 25)
    need = L.fg_lars_adam_workspace_bytes(good, 2)
    F32, F16 = fg.GRAD_F32, fg.GRAD_F16_SCALED
    for first, count in ((-1, 1), (0, 0), (1, 2), (2, 1)):
        assert L.lars_adam_norms(good, 2, first, count, ref(p), F32, 1.0, sc, ws, need,
                                 None) == fg.FG_EINVAL
    assert L.lars_adam_norms(good, 2, 0, 2, ref(p), 2, 1.0, sc, ws, need, None) == fg.FG_EINVAL
    for inv in (0.0, -1.0, float("nan"), float("inf")):
        assert L.lars_adam_norms(good, 2, 0, 2, ref(p), F16, inv, sc, ws, need,
                                 None) == fg.FG_EINVAL
    assert L.lars_adam_norms(good, 2, 0, 2, ref(p), F32, 1.0, sc, ws, need - 4,
                             None) == fg.FG_EWORKSPACE
    # an fp16 gradient needs 8-byte alignment, an fp32 one 16
    g8 = (fg.OptTensor * 1)(layer(FAKE, (4 << 16) + 8))
    assert L.lars_adam_norms(g8, 1, 0, 1, ref(p), F32, 1.0, sc, ws, need, None) == fg.FG_EINVAL
    g4 = (fg.OptTensor * 1)(layer(FAKE, (4 << 16) + 4))
    assert L.lars_adam_norms(g4, 1, 0, 1, ref(p), F16, 0.5, sc, ws, need, None) == fg.FG_EINVAL
    # no norms on this workspace yet: the apply is refused before any launch
    assert L.lars_adam_apply(good, 2, 0, 2, ref(p), F32, 1.0, None, 0, sc, ws, need,
                             None) == fg.FG_EINVAL
    assert L.lars_adam_apply(good, 2, 0, 2, ref(p), F32, 1.0, None, 2, sc, ws, need,
                             None) == fg.FG_EINVAL
    for first, count in ((-1, 1), (0, 0), (1, 2)):
        assert L.lars_adam_apply(good, 2, first, count, ref(p), F32, 1.0, None, 0, sc, ws,
                                 need, None) == fg.FG_EINVAL


def test_dense_glue_argument_checks(L):
    """Huber head, pooling and channel slice copies reject bad arguments
    before touching the device."""
    a, b, g = FAKE, FAKE + (1 << 24), FAKE + (1 << 25)
    E, U = fg.FG_EINVAL, fg.FG_EUNSUPPORTED
    assert L.huber_head_grad(a, b, 0, 1.0, 10.0, g, None) == E
    assert L.huber_head_grad(a, b, 64, 1.0, 0.0, g, None) == E
    assert L.huber_head_grad(a, b, 64, 1.0, -1.0, g, None) == E
    assert L.huber_head_grad(a, b, 64, float("nan"), 10.0, g, None) == E
    assert L.huber_head_grad(a, b, 64, 1.0, 10.0, a + 64, None) == E   # dy inside y
    assert L.avg_pool2d_fwd(a, 1, 5, 4, 8, b, None) == U               # odd H
    assert L.avg_pool2d_fwd(a, 1, 4, 4, 12, b, None) == U              # C % 8
    assert L.avg_pool2d_fwd(a + 8, 1, 4, 4, 8, b, None) == U           # alignment
    assert L.avg_pool2d_fwd(a, 0, 4, 4, 8, b, None) == E
    assert L.avg_pool2d_fwd(a, 1, 4, 4, 8, a + 64, None) == E          # overlap
    assert L.avg_pool2d_bwd(a, None, 1, 4, 4, 8, a + 32, None) == E    # dx over dy
    assert L.avg_pool2d_bwd(a, g, 1, 4, 4, 8, g + 64, None) == E       # dx over gate
    assert L.channel_slice_copy(a, 64, None, 0, b, 64, 10, 72, 0, None) == E   # nch > ld
    assert L.channel_slice_copy(a, 64, None, 0, b, 64, 0, 8, 0, None) == E
    assert L.channel_slice_copy(a, 60, None, 0, b, 64, 10, 8, 0, None) == U
    assert L.channel_slice_copy(a, 64, None, 0, b, 64, 10, 12, 0, None) == U
    assert L.channel_slice_copy(a + 2, 64, None, 0, b, 64, 10, 8, 0, None) == U
    assert L.channel_slice_copy(a, 64, None, 0, a + 16, 64, 10, 8, 0, None) == E  # spans overlap
    assert L.channel_slice_copy(a, 64, g, 64, g + 128, 64, 10, 8, 0, None) == E
    assert L.channel_slice_copy(a, 1 << 20, None, 0, b, 64, 1 << 12, 8, 0, None) == U


def test_strided_output_checks(L):
    """Pixel strides: honoured for a pass's output and for x where the
    forward pass and the kernel gradient read it; at least the channel
    count, a multiple of 8, a 16-byte aligned pointer; an input and output
    slice of one buffer must not share channels; the K = 1 head takes
    neither strides nor the accumulate epilogue. All refused before any
    launch (nothing below is dereferenced)."""
    ref = ctypes.byref
    x, w, y = FAKE, FAKE + (1 << 20), FAKE + (1 << 26)
    mk = lambda **k: fg.ConvDesc.make(2, 8, 8, 16, 16, 3, 3, 1, 1, **k)
    fwd = lambda d, out=y, epi=0: L.conv2d_fwd(ref(d), x, w, out, epi, None, None, 0, None)
    bwd = lambda d, out=y, epi=0: L.conv2d_bwd_data(ref(d), x, w, out, epi, None, None, 0,
                                                   None)
    assert fwd(mk(y_ld=8)) == fg.FG_EINVAL             # below the channel count
    assert fwd(mk(y_ld=20)) == fg.FG_EUNSUPPORTED      # not a multiple of 8
    assert fwd(mk(y_ld=24), out=y + 8) == fg.FG_EUNSUPPORTED   # output not 16-byte aligned
    assert fwd(mk(x_ld=20)) == fg.FG_EUNSUPPORTED      # input stride not a multiple of 8
    assert fwd(mk(x_ld=8)) == fg.FG_EINVAL             # input stride below the channel count
    # input channels 0..15 and output channels 8..23 of one buffer at stride 32
    assert fwd(mk(x_ld=32, y_ld=32), out=x + 16) == fg.FG_EINVAL
    # output channels 16..31 but at stride 40: the slices interleave and collide
    assert fwd(mk(x_ld=32, y_ld=40), out=x + 32) == fg.FG_EINVAL
    assert bwd(mk(y_ld=24)) == fg.FG_EUNSUPPORTED      # strided dy (an input)
    assert bwd(mk(x_ld=8)) == fg.FG_EINVAL
    assert fwd(mk(x_ld=-8)) == fg.FG_EINVAL
    wgt = lambda d: L.conv2d_bwd_weight(ref(d), x, FAKE + (1 << 24), y, None, 0, None)
    assert wgt(mk(x_ld=20)) == fg.FG_EUNSUPPORTED
    assert wgt(mk(x_ld=8)) == fg.FG_EINVAL
    assert wgt(mk(y_ld=24)) == fg.FG_EUNSUPPORTED       # strided dy
    # at stride 4096 the output's span (127 pixels * 4096 + 16 elements, ~1 MiB)
    # from 64 KiB past x reaches the weights at 1 MiB; dense, it would not
    assert bwd(mk(x_ld=4096), out=x + (1 << 16)) == fg.FG_EINVAL
    head = lambda **k: fg.ConvDesc.make(2, 8, 8, 16, 1, 1, 1, 1, 0, **k)
    assert fwd(head(y_ld=8)) == fg.FG_EUNSUPPORTED
    assert fwd(head(), epi=fg.EPI_ACC) == fg.FG_EUNSUPPORTED
    assert bwd(head(x_ld=24)) == fg.FG_EUNSUPPORTED
    assert fwd(head(x_ld=24)) == fg.FG_EUNSUPPORTED
    assert wgt(head(x_ld=24)) == fg.FG_EUNSUPPORTED


def test_gate_must_not_overlap_the_output(L):
    """A ReLU-gradient gate that partly overlaps the output is refused (a
    workgroup could overwrite gate values another one has yet to read)."""
    d = _desc()
    ref = ctypes.byref
    x, w, y = FAKE, FAKE + (1 << 20), FAKE + (1 << 22)
    assert L.conv2d_fwd(ref(d), x, w, y, fg.EPI_GATE, y + 64, None, 0,
                        None) == fg.FG_EINVAL
    assert L.conv2d_fwd(ref(d), x, w, y, fg.EPI_GATE, y - 64, None, 0,
                        None) == fg.FG_EINVAL
    dy, dx = FAKE, FAKE + (1 << 22)
    assert L.conv2d_bwd_data(ref(d), dy, w, dx, fg.EPI_GATE, dx + 2, None, 0,
                             None) == fg.FG_EINVAL
    t = fg.ConvDesc.make(2, 8, 8, 16, 16, 4, 4, 2, 1)
    yt = FAKE + (1 << 23)
    assert L.conv_transpose2d_fwd(ref(t), FAKE, w, yt, fg.EPI_GATE, yt + 128, None,
                                  0, None) == fg.FG_EINVAL


def test_flags_clear_and_host_helpers_validate(L):
    assert L.grad_flags_clear(None, 4, None) == fg.FG_EINVAL
    assert L.grad_flags_clear(FAKE, 0, None) == fg.FG_EINVAL
    # disarming the profiling events needs no device
    assert L.fg_profile_next_launch(None, None) == fg.FG_OK
    applied = ctypes.c_int32(7)
    for bad in (fg.LossScaleState(2.0 ** 15, 0, 0, 1.0, 2.0 ** 24),      # interval
                fg.LossScaleState(0.5, 0, 10, 1.0, 2.0 ** 24),          # below s_min
                fg.LossScaleState(2.0 ** 25, 0, 10, 1.0, 2.0 ** 24),    # above s_max
                fg.LossScaleState(1.0, 0, 10, 0.0, 2.0 ** 24)):         # s_min 0
        before = bytes(bad)
        assert L.fg_loss_scale_update(ctypes.byref(bad), 0,
                                      ctypes.byref(applied)) == fg.FG_EINVAL
        assert bytes(bad) == before and applied.value == 7
    out = ctypes.c_double()
    for bad, k in ((fg.LRScheduleParams(1e-4, 1e-3, 10, 0, 1.0), -1),
                   (fg.LRScheduleParams(-1e-4, 1e-3, 10, 0, 1.0), 0),
                   (fg.LRScheduleParams(1e-4, 1e-3, -1, 0, 1.0), 0),
                   (fg.LRScheduleParams(1e-4, 1e-3, 10, 0, 0.0), 0)):
        assert L.fg_lr_at(ctypes.byref(bad), k, ctypes.byref(out)) == fg.FG_EINVAL


def test_noalloc_kernel_gradient_validates_before_any_device_call(L):
    d = _desc()
    ref = ctypes.byref
    assert L.conv2d_bwd_weight_noalloc(None, FAKE, FAKE + (1 << 20), FAKE + (1 << 22),
                                       None) == fg.FG_EINVAL
    assert L.conv2d_bwd_weight_noalloc(ref(d), None, FAKE + (1 << 20), FAKE + (1 << 22),
                                       None) == fg.FG_EINVAL
    # dW aliasing x
    assert L.conv2d_bwd_weight_noalloc(ref(d), FAKE, FAKE + (1 << 20), FAKE,
                                       None) == fg.FG_EINVAL
    assert L.conv2d_bwd_weight_noalloc(ref(_desc(c=12)), FAKE, FAKE + (1 << 20),
                                       FAKE + (1 << 22), None) == fg.FG_EUNSUPPORTED


def test_random_shape_sweep_reaches_every_kernel_family(L):
    """The seeded shapes of the GPU sweep take every convolution kernel
    family, non-square kernels, strided input gradients and empty phases."""
    import test_gpu_sweep
    test_gpu_sweep.check_coverage()


def test_plain_c_consumer_builds_and_plans(L, tmp_path):
    """The header compiles as C11 (gcc, warnings as errors) and a C program
    linked against the library gets the oracle's group plan, the output
    sizes, the workspace and kernel the binding reports, and FG_EINVAL for
    null pointers; no GPU is touched."""
    import shutil
    import subprocess
    import numpy as np
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "abi_consumer")
    libdir = os.path.dirname(fg.LIB_PATH)
    subprocess.run([gcc, "-std=c11", "-Wall", "-Wextra", "-Werror",
                    "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include",
                    os.path.join(ROOT, "tests", "c_consumer", "abi_consumer.c"),
                    "-L", libdir, "-lfcngrad", f"-Wl,-rpath,{libdir}", "-o", exe],
                   check=True, timeout=120)
    rng = np.random.default_rng(11)
    numels = [int(v) for v in rng.integers(1, 200_000, size=40)]
    cap, align = 1 << 20, 256
    r = subprocess.run([exe, str(cap), str(align)], input=" ".join(map(str, numels)),
                       capture_output=True, text=True, timeout=60, check=True)
    lines = r.stdout.splitlines()
    plan = G.plan_groups(numels, cap, align)
    assert lines[0] == f"plan {len(plan)}"
    want = {}
    for gi, p in enumerate(plan):
        for m, off in zip(p["members"], p["offsets"]):
            want[m] = f"{gi} {off}"
    assert lines[1:1 + len(numels)] == [want[i] for i in range(len(numels))]
    rest = lines[1 + len(numels):]
    assert rest[:len(plan)] == [str(p["numel"]) for p in plan]
    kv = dict(ln.split(" ", 1) for ln in rest[len(plan):])
    d = fg.ConvDesc.make(4, 256, 256, 256, 512, 3, 3, 2, 1)
    assert kv["out_dims"] == "128 128 256 256"
    assert kv["ws"] == str(fg.workspace_bytes(d, fg.OP_BWD_WEIGHT))
    assert kv["kernel"] == fg.kernel_name(d, fg.OP_BWD_WEIGHT)
    assert kv["einval"] == "OK"
    assert kv["status"] == fg.status_string(fg.FG_EUNSUPPORTED)


def test_mfma_loop_argument_checks(L):
    """fg_mfma_loop rejects its bad arguments on the host (nothing is
    launched; the pointer below is never dereferenced)."""
    ok = fg.FG_EINVAL
    assert L.fg_mfma_loop(None, 1, 1, 0, None) == ok
    assert L.fg_mfma_loop(FAKE, 0, 1, 0, None) == ok
    assert L.fg_mfma_loop(FAKE, 1, 0, 0, None) == ok
    assert L.fg_mfma_loop(FAKE, 1, 1, 2, None) == ok
    assert L.fg_mfma_loop(FAKE, 1 << 15, (fg.MFMA_LOOP_MAX_WORK >> 15) + 1, 0, None) == ok
    import torch
    with pytest.raises(ValueError):
        fg.mfma_loop(torch.empty(255, dtype=torch.float32), 1, 1)
    with pytest.raises(ValueError):
        fg.mfma_loop(torch.empty(256, dtype=torch.float16), 1, 1)
