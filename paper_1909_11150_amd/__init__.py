"""Python binding of libfcngrad (fp16 FCN training-step hot path, gfx950).

Argument marshalling only: every call forwards device pointers of torch
tensors and the current HIP stream to the C ABI declared in
``include/fcngrad.h``; all arithmetic runs in the library's HIP kernels.
PyTorch provides device memory and streams. The library is loaded from
this directory; a missing library raises ``LibraryNotBuilt`` — there is no
fallback path.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfcngrad.so")

FG_OK, FG_EINVAL, FG_EUNSUPPORTED, FG_EWORKSPACE, FG_ELAUNCH = range(5)
EPI_NONE, EPI_RELU, EPI_GATE, EPI_ACC = 0, 1, 2, 3
OP_FWD, OP_BWD_DATA, OP_BWD_WEIGHT, OP_CONVT = 0, 1, 2, 3
MAX_SEGMENTS = 64
GRAD_F32, GRAD_F16_SCALED = 0, 1

ENTRY_POINTS = (
    "conv2d_fwd", "conv2d_bwd_data", "conv2d_bwd_weight",
    "conv2d_bwd_weight_checked", "conv_transpose2d_fwd", "grad_group_pack", "grad_unscale_check",
    "grad_group_unpack", "l2_head_grad", "relu_backward",
    "fg_conv_workspace_bytes", "fg_conv_out_dims", "grad_group_plan",
    "fg_conv_kernel_name", "fg_status_string",
    "lars_adam_update", "lars_adam_norms", "lars_adam_apply",
    "fg_lars_adam_workspace_bytes",
    "huber_head_grad", "avg_pool2d_fwd", "avg_pool2d_bwd", "channel_slice_copy",
    "grad_flags_clear", "fg_loss_scale_update", "fg_lr_at", "fg_profile_next_launch",
    "conv2d_bwd_weight_noalloc", "fg_mfma_loop",
)
MFMA_LOOP_MAX_WORK = 1 << 28  # blocks * iters accepted by fg_mfma_loop
MFMA_LOOP_FLOPS_PER_BLOCK_ITER = 1 << 20
NOALLOC_SCRATCH_BYTES = 64 << 20


class OptTensor(ctypes.Structure):
    """fg_opt_tensor: one layer's device arrays for lars_adam_update."""
    _fields_ = [("w32", ctypes.c_uint64), ("w16", ctypes.c_uint64),
                ("m", ctypes.c_uint64), ("v", ctypes.c_uint64),
                ("g", ctypes.c_uint64), ("numel", ctypes.c_uint64)]


class OptParams(ctypes.Structure):
    """fg_opt_params."""
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float)]


class LossScaleState(ctypes.Structure):
    """fg_loss_scale: backoff loss-scale state."""
    _fields_ = [("scale", ctypes.c_double), ("clean", ctypes.c_int32),
                ("interval", ctypes.c_int32), ("s_min", ctypes.c_double),
                ("s_max", ctypes.c_double)]


class LRScheduleParams(ctypes.Structure):
    """fg_lr_schedule."""
    _fields_ = [("base", ctypes.c_double), ("peak", ctypes.c_double),
                ("warmup", ctypes.c_int64), ("every", ctypes.c_int64),
                ("rate", ctypes.c_double)]


class LibraryNotBuilt(RuntimeError):
    pass


class FgError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn}: {status_string(status)}")


class ConvDesc(ctypes.Structure):
    """fg_conv_desc. x_ld / y_ld: pixel strides of the x- and y-shaped
    tensors (0: dense), honoured where that tensor is the pass's output and
    for x where the forward pass and the kernel gradient read it."""
    _fields_ = [(f, ctypes.c_int32) for f in
                ("n", "h", "w", "c", "k", "r", "s", "stride_h", "stride_w",
                 "pad_h", "pad_w", "x_ld", "y_ld")]

    @classmethod
    def make(cls, n, h, w, c, k, r, s, stride=1, pad=0, x_ld=0, y_ld=0):
        return cls(n, h, w, c, k, r, s, stride, stride, pad, pad, x_ld, y_ld)


class Segment(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_uint64), ("numel", ctypes.c_uint64),
                ("offset", ctypes.c_uint64)]


_lib = None


def lib():
    """Load libfcngrad.so (once) and declare every entry point."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise LibraryNotBuilt(
            f"{LIB_PATH} is missing; build it with "
            "`python -m paper_1909_11150_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
    pdesc = ctypes.POINTER(ConvDesc)
    pseg = ctypes.POINTER(Segment)
    sigs = {
        "conv2d_fwd": [pdesc, vp, vp, vp, i32, vp, vp, sz, vp],
        "conv2d_bwd_data": [pdesc, vp, vp, vp, i32, vp, vp, sz, vp],
        "conv2d_bwd_weight": [pdesc, vp, vp, vp, vp, sz, vp],
        "conv2d_bwd_weight_checked": [pdesc, vp, vp, vp, vp, vp, sz, vp],
        "conv2d_bwd_weight_noalloc": [pdesc, vp, vp, vp, vp],
        "conv_transpose2d_fwd": [pdesc, vp, vp, vp, i32, vp, vp, sz, vp],
        "grad_group_pack": [pseg, i32, vp, u64, vp],
        "grad_unscale_check": [vp, u64, ctypes.c_float, vp, vp, vp],
        "grad_group_unpack": [vp, u64, pseg, i32, vp],
        "l2_head_grad": [vp, vp, u64, ctypes.c_double, vp, vp],
        "relu_backward": [vp, vp, u64, vp, vp],
        "grad_flags_clear": [vp, i32, vp],
        "fg_loss_scale_update": [ctypes.POINTER(LossScaleState), i32, ctypes.POINTER(i32)],
        "fg_lr_at": [ctypes.POINTER(LRScheduleParams), ctypes.c_int64,
                     ctypes.POINTER(ctypes.c_double)],
        "fg_profile_next_launch": [vp, vp],
        "fg_mfma_loop": [vp, i32, i32, i32, vp],
        "huber_head_grad": [vp, vp, u64, ctypes.c_double, ctypes.c_double, vp, vp],
        "avg_pool2d_fwd": [vp, i32, i32, i32, i32, vp, vp],
        "avg_pool2d_bwd": [vp, vp, i32, i32, i32, i32, vp, vp],
        "channel_slice_copy": [vp, i32, vp, i32, vp, i32, ctypes.c_int64, i32, i32, vp],
        "fg_conv_out_dims": [pdesc, ctypes.c_int, ctypes.POINTER(i32),
                             ctypes.POINTER(i32)],
        "grad_group_plan": [ctypes.POINTER(u64), i32, u64, ctypes.c_uint32,
                            ctypes.c_uint32, ctypes.POINTER(i32),
                            ctypes.POINTER(u64), ctypes.POINTER(i32),
                            ctypes.POINTER(u64)],
    }
    for name, args in sigs.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    L.lars_adam_update.argtypes = [ctypes.POINTER(OptTensor), i32,
                                   ctypes.POINTER(OptParams), vp, i32, vp, vp, sz, vp]
    L.lars_adam_update.restype = ctypes.c_int
    L.lars_adam_norms.argtypes = [ctypes.POINTER(OptTensor), i32, i32, i32,
                                  ctypes.POINTER(OptParams), i32, ctypes.c_float, vp,
                                  vp, sz, vp]
    L.lars_adam_norms.restype = ctypes.c_int
    L.lars_adam_apply.argtypes = [ctypes.POINTER(OptTensor), i32, i32, i32,
                                  ctypes.POINTER(OptParams), i32, ctypes.c_float, vp,
                                  i32, vp, vp, sz, vp]
    L.lars_adam_apply.restype = ctypes.c_int
    L.fg_lars_adam_workspace_bytes.argtypes = [ctypes.POINTER(OptTensor), i32]
    L.fg_lars_adam_workspace_bytes.restype = ctypes.c_size_t
    L.fg_conv_workspace_bytes.argtypes = [pdesc, ctypes.c_int]
    L.fg_conv_workspace_bytes.restype = ctypes.c_size_t
    L.fg_conv_kernel_name.argtypes = [pdesc, ctypes.c_int]
    L.fg_conv_kernel_name.restype = ctypes.c_char_p
    L.fg_status_string.argtypes = [ctypes.c_int]
    L.fg_status_string.restype = ctypes.c_char_p
    _lib = L
    return L


def status_string(status):
    return lib().fg_status_string(status).decode()


def _check(fn, status):
    if status != FG_OK:
        raise FgError(fn, status)


def _p(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libfcngrad must be contiguous")
    return t.data_ptr()


def _s(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream


# ---- convolution passes ---------------------------------------------------
def kernel_name(desc, op):
    """Main kernel the pass launches for this shape (for grouping timings)."""
    return lib().fg_conv_kernel_name(ctypes.byref(desc), op).decode()


def workspace_bytes(desc, op):
    return lib().fg_conv_workspace_bytes(ctypes.byref(desc), op)


def out_dims(desc, transpose=False):
    p, q = ctypes.c_int32(), ctypes.c_int32()
    _check("fg_conv_out_dims", lib().fg_conv_out_dims(
        ctypes.byref(desc), int(transpose), ctypes.byref(p), ctypes.byref(q)))
    return p.value, q.value


def _ws(ws):
    return (None, 0) if ws is None else (ws.data_ptr(), ws.numel() * ws.element_size())


def conv2d_fwd(desc, x, w, y, epi=EPI_NONE, gate=None, ws=None, stream=None):
    wp, wb = _ws(ws)
    _check("conv2d_fwd", lib().conv2d_fwd(
        ctypes.byref(desc), _p(x), _p(w), _p(y), epi, _p(gate), wp, wb, _s(stream)))


def conv2d_bwd_data(desc, dy, w, dx, epi=EPI_NONE, gate=None, ws=None,
                    stream=None):
    wp, wb = _ws(ws)
    _check("conv2d_bwd_data", lib().conv2d_bwd_data(
        ctypes.byref(desc), _p(dy), _p(w), _p(dx), epi, _p(gate), wp, wb,
        _s(stream)))


def conv2d_bwd_weight(desc, x, dy, dw, ws=None, stream=None):
    wp, wb = _ws(ws)
    _check("conv2d_bwd_weight", lib().conv2d_bwd_weight(
        ctypes.byref(desc), _p(x), _p(dy), _p(dw), wp, wb, _s(stream)))


def conv2d_bwd_weight_noalloc(desc, x, dy, dw, stream=None):
    """conv2d_bwd_weight with its split partials in the library's static
    scratch: no workspace argument, nothing allocated."""
    _check("conv2d_bwd_weight_noalloc", lib().conv2d_bwd_weight_noalloc(
        ctypes.byref(desc), _p(x), _p(dy), _p(dw), _s(stream)))


def conv2d_bwd_weight_checked(desc, x, dy, dw, found_nonfinite, ws=None,
                              stream=None):
    """conv2d_bwd_weight that also sets the device int32 found_nonfinite to 1
    if a written dW element is +-inf or NaN; dw may be a view into a group
    buffer (zero-copy pack)."""
    wp, wb = _ws(ws)
    _check("conv2d_bwd_weight_checked", lib().conv2d_bwd_weight_checked(
        ctypes.byref(desc), _p(x), _p(dy), _p(dw), _p(found_nonfinite), wp, wb,
        _s(stream)))


def opt_tensors(w32, w16, m, v, g):
    """fg_opt_tensor array for lists of per-layer torch tensors."""
    n = len(w32)
    arr = (OptTensor * n)(*[OptTensor(w32[i].data_ptr(), w16[i].data_ptr(),
                                      m[i].data_ptr(), v[i].data_ptr(),
                                      g[i].data_ptr(), w32[i].numel())
                            for i in range(n)])
    return arr


def lars_adam_workspace_bytes(tensors):
    return lib().fg_lars_adam_workspace_bytes(tensors, len(tensors))


def lars_adam_update(tensors, lr, flags, step_count, ws, beta1=0.9, beta2=0.999,
                     eps=1e-8, weight_decay=1e-4, stream=None):
    """Layer-wise adaptive Adam step (see include/fcngrad.h). tensors: from
    opt_tensors(); flags: device int32 tensor of the step's group flags (or
    None); step_count: device int32 tensor of one element."""
    p = OptParams(lr, beta1, beta2, eps, weight_decay)
    wp, wb = _ws(ws)
    nf = 0 if flags is None else flags.numel()
    _check("lars_adam_update", lib().lars_adam_update(
        tensors, len(tensors), ctypes.byref(p), _p(flags), nf, _p(step_count),
        wp, wb, _s(stream)))


def lars_adam_norms(tensors, first, count, step_count, ws, grad_format=GRAD_F32,
                    grad_inv_scale=1.0, beta1=0.9, beta2=0.999, eps=1e-8,
                    weight_decay=1e-4, stream=None):
    """Partial norms of layers [first, first + count) (see include/fcngrad.h);
    the learning rate does not enter."""
    p = OptParams(0.0, beta1, beta2, eps, weight_decay)
    wp, wb = _ws(ws)
    _check("lars_adam_norms", lib().lars_adam_norms(
        tensors, len(tensors), first, count, ctypes.byref(p), grad_format,
        grad_inv_scale, _p(step_count), wp, wb, _s(stream)))


def lars_adam_apply(tensors, lr, flags, step_count, ws, grad_format=GRAD_F32,
                    grad_inv_scale=1.0, beta1=0.9, beta2=0.999, eps=1e-8,
                    weight_decay=1e-4, first=0, count=None, stream=None):
    """Update of layers [first, first + count) (default: all) once
    lars_adam_norms has covered every layer."""
    p = OptParams(lr, beta1, beta2, eps, weight_decay)
    wp, wb = _ws(ws)
    nf = 0 if flags is None else flags.numel()
    if count is None:
        count = len(tensors) - first
    _check("lars_adam_apply", lib().lars_adam_apply(
        tensors, len(tensors), first, count, ctypes.byref(p), grad_format, grad_inv_scale,
        _p(flags), nf, _p(step_count), wp, wb, _s(stream)))


def conv_transpose2d_fwd(desc, x, w, y, epi=EPI_NONE, gate=None, ws=None,
                         stream=None):
    wp, wb = _ws(ws)
    _check("conv_transpose2d_fwd", lib().conv_transpose2d_fwd(
        ctypes.byref(desc), _p(x), _p(w), _p(y), epi, _p(gate), wp, wb,
        _s(stream)))


# ---- gradient path --------------------------------------------------------
def _segments(tensors, offsets):
    arr = (Segment * len(tensors))()
    for i, (t, off) in enumerate(zip(tensors, offsets)):
        arr[i] = Segment(_p(t), t.numel(), off)
    return arr


def grad_group_pack(srcs, offsets, group, stream=None):
    segs = _segments(srcs, offsets)
    _check("grad_group_pack", lib().grad_group_pack(
        segs, len(srcs), _p(group), group.numel(), _s(stream)))


def grad_unscale_check(group, inv_scale, out_f32, flag, numel=None,
                       stream=None):
    n = group.numel() if numel is None else numel
    _check("grad_unscale_check", lib().grad_unscale_check(
        _p(group), n, float(inv_scale), _p(out_f32), _p(flag), _s(stream)))


def grad_group_unpack(group_f32, dsts, offsets, stream=None):
    segs = _segments(dsts, offsets)
    _check("grad_group_unpack", lib().grad_group_unpack(
        _p(group_f32), group_f32.numel(), segs, len(dsts), _s(stream)))


def l2_head_grad(y, t, scale, dy, stream=None):
    _check("l2_head_grad", lib().l2_head_grad(
        _p(y), _p(t), y.numel(), float(scale), _p(dy), _s(stream)))


def huber_head_grad(y, t, scale, delta, dy, stream=None):
    """dy = fp16(scale * clamp(y - t, -delta, delta)); scale = S / numel for
    the loss-scaled mean Huber loss."""
    _check("huber_head_grad", lib().huber_head_grad(
        _p(y), _p(t), y.numel(), float(scale), float(delta), _p(dy), _s(stream)))


def avg_pool2d_fwd(x, y, stream=None):
    """2x2 stride-2 mean pooling of an N x H x W x C fp16 tensor."""
    n, h, w, c = x.shape
    _check("avg_pool2d_fwd", lib().avg_pool2d_fwd(_p(x), n, h, w, c, _p(y), _s(stream)))


def avg_pool2d_bwd(dy, dx, gate=None, stream=None):
    """Gradient of avg_pool2d_fwd into dx (the forward input's shape),
    zero where gate <= 0 if a gate is given."""
    n, h, w, c = dx.shape
    _check("avg_pool2d_bwd", lib().avg_pool2d_bwd(
        _p(dy), _p(gate), n, h, w, c, _p(dx), _s(stream)))


def channel_slice_copy(src, src_ld, dst, dst_ld, npix, nch, gate=None, gate_ld=0,
                       accumulate=False, stream=None):
    """Per pixel, nch channels from src (pixel stride src_ld) to dst (pixel
    stride dst_ld); src, dst, gate: tensors or device addresses (a channel
    offset is an address offset)."""
    def a(x):
        return None if x is None else (x if isinstance(x, int) else x.data_ptr())
    _check("channel_slice_copy", lib().channel_slice_copy(
        a(src), src_ld, a(gate), gate_ld, a(dst), dst_ld, npix, nch, int(accumulate),
        _s(stream)))


def grad_flags_clear(flags, stream=None):
    """Zero a device int32 tensor of non-finite flags with a library kernel."""
    _check("grad_flags_clear", lib().grad_flags_clear(_p(flags), flags.numel(),
                                                      _s(stream)))


def profile_next_launch(start, stop):
    """Arm two torch.cuda.Events (timing enabled) around the main kernel of
    the next convolution call on this thread; None, None disarms."""
    for e in (start, stop):  # torch creates an event at its first record
        if e is not None and not e.cuda_event:
            e.record()
    a = None if start is None else start.cuda_event
    b = None if stop is None else stop.cuda_event
    _check("fg_profile_next_launch", lib().fg_profile_next_launch(a, b))


def mfma_loop(out, blocks, iters, operands=0, stream=None):
    """Register-only MFMA chains (fg_mfma_loop): out is a float32 device
    tensor of at least blocks * 256 elements; blocks * iters * 2^20 flops."""
    if (not out.is_floating_point() or out.element_size() != 4
            or out.numel() < blocks * 256):
        raise ValueError("fg_mfma_loop needs blocks * 256 float32 outputs")
    _check("fg_mfma_loop", lib().fg_mfma_loop(_p(out), blocks, iters, operands, _s(stream)))


def loss_scale_update(state, found_nonfinite):
    """Advance a LossScaleState by one step's outcome; True if it applies."""
    applied = ctypes.c_int32()
    _check("fg_loss_scale_update", lib().fg_loss_scale_update(
        ctypes.byref(state), int(bool(found_nonfinite)), ctypes.byref(applied)))
    return bool(applied.value)


def lr_at(params, k):
    """Learning rate of applied step k under an LRScheduleParams."""
    out = ctypes.c_double()
    _check("fg_lr_at", lib().fg_lr_at(ctypes.byref(params), int(k), ctypes.byref(out)))
    return out.value


def relu_backward(dy, act, out, stream=None):
    _check("relu_backward", lib().relu_backward(
        _p(dy), _p(act), dy.numel(), _p(out), _s(stream)))


def grad_group_plan(numels, cap_bytes, align_bytes=256, elem_bytes=2):
    """Host planner in the library: returns (group_of, offset_of, group_numel)."""
    n = len(numels)
    u64a = (ctypes.c_uint64 * n)(*numels)
    gof = (ctypes.c_int32 * n)()
    oof = (ctypes.c_uint64 * n)()
    gnum = (ctypes.c_uint64 * n)()
    ng = ctypes.c_int32()
    _check("grad_group_plan", lib().grad_group_plan(
        u64a, n, cap_bytes, align_bytes, elem_bytes, gof, oof,
        ctypes.byref(ng), gnum))
    return list(gof), list(oof), list(gnum[:ng.value])
