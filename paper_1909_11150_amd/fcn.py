"""One GPU's share of a training step of the fully convolutional network.

``Chain`` sequences the library's calls for a chain of conv / transposed-conv
layers (Section 6.2, Figure workflow (B): encoder-decoder): the forward pass
with fused ReLUs, the loss-scaled L2 head gradient, the backward pass with
fused ReLU gradients, and — per complete gradient group, in backward
completion order — fusion-buffer pack, unscale with overflow check and
unpack to fp32 master gradients (Section 4.2 Grouping; Section 6.2 loss
scaling) — and, with an optimizer, the layer-wise adaptive Adam update of
fp32 master weights under a backoff loss scale (Section 6.2). Device memory
comes from torch; every step is a libfcngrad call.

Layers are duck-typed: ``kind`` ("conv" | "convT"), ``x_shape``/``y_shape``
(NHWC), ``r``, ``s``, ``stride``, ``pad``, ``relu`` and ``w_shape``.
"""
import ctypes
from collections import namedtuple

import torch

from . import (EPI_GATE, EPI_NONE, EPI_RELU, OP_BWD_DATA, OP_BWD_WEIGHT,
               OP_CONVT, OP_FWD, ConvDesc, FgError, LossScaleState, LRScheduleParams,
               OptParams, Segment, grad_flags_clear, loss_scale_update, lr_at,
               profile_next_launch,
               GRAD_F16_SCALED, GRAD_F32, kernel_name, lib,
               conv2d_bwd_data, conv2d_bwd_weight, conv2d_bwd_weight_checked,
               conv2d_fwd,
               conv_transpose2d_fwd, grad_group_pack, grad_group_plan,
               grad_group_unpack, grad_unscale_check, l2_head_grad,
               lars_adam_update, lars_adam_workspace_bytes, opt_tensors,
               relu_backward, workspace_bytes)

F16 = torch.float16


def fwd_desc(L):
    """Descriptor of the layer's forward op (convT: its own input/output)."""
    n, h, w, c = L.x_shape
    k = L.y_shape[3]
    return ConvDesc.make(n, h, w, c, k, L.r, L.s, L.stride, L.pad)


def convt_dx_desc(L):
    """Input gradient of a transposed conv: a forward conv of dy (the big
    image) with Wt read as KRSC (K = C_in, C = C_out)."""
    n, ho, wo, co = L.y_shape
    ci = L.x_shape[3]
    return ConvDesc.make(n, ho, wo, co, ci, L.r, L.s, L.stride, L.pad)


def convt_dw_desc(L):
    """Kernel gradient of a transposed conv: the conv kernel gradient with
    x := dy (big image, C = C_out channels) and dy := x (K = C_in)."""
    return convt_dx_desc(L)


def chain_workspace_bytes(layers):
    """Largest workspace any pass of any layer needs (one shared buffer:
    the passes run in stream order)."""
    ws = 0
    for L in layers:
        if L.kind == "conv":
            d = fwd_desc(L)
            for op in (OP_FWD, OP_BWD_DATA, OP_BWD_WEIGHT):
                ws = max(ws, workspace_bytes(d, op))
        else:
            ws = max(ws, workspace_bytes(fwd_desc(L), OP_CONVT))
            d = convt_dx_desc(L)
            for op in (OP_FWD, OP_BWD_WEIGHT):
                ws = max(ws, workspace_bytes(d, op))
    return ws


class LossScaler:
    """Backoff loss scaling (Section 6.2: the loss is scaled before the
    gradient computation, with OpenSeq2Seq's adaptive strategy): the state
    of the library's fg_loss_scale_update. A step whose gradients hold a
    non-finite value is not applied; it halves the scale (not below s_min)
    and restarts the count of clean steps. After `interval` clean steps in a
    row the scale doubles (not above s_max)."""

    def __init__(self, scale=2.0 ** 15, interval=2000, s_min=1.0, s_max=2.0 ** 24):
        if interval < 1 or not 0 < s_min <= scale <= s_max:
            raise ValueError("need interval >= 1 and 0 < s_min <= scale <= s_max")
        self._st = LossScaleState(float(scale), 0, int(interval), float(s_min),
                                  float(s_max))

    scale = property(lambda self: self._st.scale)
    clean = property(lambda self: self._st.clean)
    interval = property(lambda self: self._st.interval)
    s_min = property(lambda self: self._st.s_min)
    s_max = property(lambda self: self._st.s_max)

    def update(self, found_nonfinite):
        """Record one step's outcome; returns whether its update applied."""
        return loss_scale_update(self._st, found_nonfinite)


class LRSchedule:
    """Learning rate per applied step (Section 6.2), evaluated by the
    library's fg_lr_at: a linear warm-up from `base` to `peak` (the paper's
    N * base for N ranks) over `warmup` steps, then a staircase decay by
    `rate` every `every` steps (every = 0: none). The step index counts
    applied updates from 0."""

    def __init__(self, base=1e-4, peak=None, warmup=0, every=0, rate=1.0):
        self.base = float(base)
        self.peak = self.base if peak is None else float(peak)
        self.warmup, self.every, self.rate = int(warmup), int(every), float(rate)
        if self.warmup < 0 or self.every < 0 or self.base < 0 or self.peak < 0:
            raise ValueError("negative schedule parameter")
        self._p = LRScheduleParams(self.base, self.peak, self.warmup, self.every,
                                   self.rate)

    def __call__(self, k):
        return lr_at(self._p, k)


class AdamLARS:
    """Hyperparameters of the layer-wise adaptive Adam update (Section 6.2:
    Adam with beta1 0.9, beta2 0.999; L2 weight decay 1e-4). lr: a float or
    a schedule called with the number of applied steps."""

    def __init__(self, lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8,
                 weight_decay=1e-4):
        self.lr = lr
        self.beta1, self.beta2 = float(beta1), float(beta2)
        self.eps, self.weight_decay = float(eps), float(weight_decay)

    def lr_at(self, k):
        return float(self.lr(k)) if callable(self.lr) else float(self.lr)


class Chain:
    def __init__(self, layers, weights, x, device="cuda", loss_scale=2.0 ** 15,
                 group_cap_bytes=None, group_align_bytes=256, stream=None,
                 zero_copy=False, optimizer=None, scaler=None):
        """zero_copy (with groups): each layer's fp16 dW lives in its slot of
        its group buffer, written there by conv2d_bwd_weight_checked (which
        also raises the group's non-finite flag), so no pack is needed; the
        gaps between slots are zeroed once here.
        optimizer (an AdamLARS; needs groups): the step ends with the update
        of fp32 master weights (initialised from the given weights), their
        Adam moments and the fp16 working weights the passes read; a step
        with a flagged group is skipped on the device.
        scaler (a LossScaler): the loss scale follows the flags of each step
        (loss_scale is then taken from it)."""
        self.layers = list(layers)
        self.zero_copy = bool(zero_copy)
        self.dev = torch.device(device)
        self.stream = stream
        self.scaler = scaler
        self.loss_scale = float(scaler.scale if scaler is not None else loss_scale)
        self.w = [torch.as_tensor(w).to(self.dev).contiguous() for w in weights]
        self.x = torch.as_tensor(x).to(self.dev).contiguous()
        nl = len(self.layers)
        self.acts = [self.x] + [torch.empty(L.y_shape, dtype=F16, device=self.dev)
                                for L in self.layers]
        # g[i]: gradient w.r.t. the pre-activation output of layer i-1 (g[0]
        # is the input gradient of the network)
        self.g = [torch.empty(L.x_shape, dtype=F16, device=self.dev)
                  for L in self.layers] + \
                 [torch.empty(self.layers[-1].y_shape, dtype=F16, device=self.dev)]
        self.dw = [torch.empty(L.w_shape, dtype=F16, device=self.dev)
                   for L in self.layers]
        self.ws = torch.empty(max(chain_workspace_bytes(self.layers), 16),
                              dtype=torch.uint8, device=self.dev)
        self.groups = None
        self.group_cap_bytes = group_cap_bytes
        if group_cap_bytes is not None:
            self._plan_groups(group_cap_bytes, group_align_bytes)
        self._nl = nl
        self.opt = optimizer
        self.applied = 0  # updates applied (host count, known after a step)
        if optimizer is not None:
            self._init_optimizer()

    # ---- optimizer state ----------------------------------------------------------
    def _init_optimizer(self):
        if self.groups is None:
            raise ValueError("the optimizer needs gradient groups (group_cap_bytes)")
        if any(w.dtype != F16 for w in self.w):
            raise ValueError("the optimizer writes fp16 working weights")
        f32 = torch.float32
        self.w32 = [w.to(f32).contiguous() for w in self.w]
        self.m = [torch.zeros_like(w) for w in self.w32]
        self.v = [torch.zeros_like(w) for w in self.w32]
        self.step_count = torch.zeros(1, dtype=torch.int32, device=self.dev)
        self.opt_tensors = opt_tensors(self.w32, self.w, self.m, self.v, self.master)
        self.opt_ws = torch.empty(max(lars_adam_workspace_bytes(self.opt_tensors), 16),
                                  dtype=torch.uint8, device=self.dev)

    def update(self):
        """The optimizer step on the unpacked gradients (skipped on the device
        when a group flag is set)."""
        o = self.opt
        lars_adam_update(self.opt_tensors, o.lr_at(self.applied), self.flags,
                         self.step_count, self.opt_ws, o.beta1, o.beta2, o.eps,
                         o.weight_decay, stream=self.stream)

    # ---- gradient groups ---------------------------------------------------
    def _plan_groups(self, cap, align):
        order = list(reversed(range(len(self.layers))))  # completion order
        numels = [self.dw[i].numel() for i in order]
        gof, oof, gnum = grad_group_plan(numels, cap, align, 2)
        groups = []
        for g, n in enumerate(gnum):
            mem = [(order[j], oof[j]) for j in range(len(order)) if gof[j] == g]
            groups.append({"members": [m for m, _ in mem],
                           "offsets": [o for _, o in mem], "numel": n})
        self.groups = groups
        alloc = torch.zeros if self.zero_copy else torch.empty
        self.gbuf16 = [alloc(g["numel"], dtype=F16, device=self.dev)
                       for g in groups]
        if self.zero_copy:  # dW tensors become views of their group slots
            for gi, g in enumerate(groups):
                for m, off in zip(g["members"], g["offsets"]):
                    n = self.dw[m].numel()
                    self.dw[m] = self.gbuf16[gi][off:off + n].view(self.dw[m].shape)
        # group of each layer's dW
        self._group_of = {m: gi for gi, g in enumerate(groups) for m in g["members"]}
        self.gbuf32 = [torch.empty(g["numel"], dtype=torch.float32, device=self.dev)
                       for g in groups]
        self.flags = torch.zeros(len(groups), dtype=torch.int32, device=self.dev)
        self.master = [torch.empty(L.w_shape, dtype=torch.float32, device=self.dev)
                       for L in self.layers]
        # the layer whose dW completes each group (last member in order)
        self._group_done_at = {g["members"][-1]: gi for gi, g in enumerate(groups)}

    def run_group(self, gi):
        g = self.groups[gi]
        if not self.zero_copy:
            grad_group_pack([self.dw[m] for m in g["members"]], g["offsets"],
                            self.gbuf16[gi], stream=self.stream)
        grad_unscale_check(self.gbuf16[gi], 1.0 / self.loss_scale,
                           self.gbuf32[gi], self.flags[gi:gi + 1],
                           stream=self.stream)
        grad_group_unpack(self.gbuf32[gi], [self.master[m] for m in g["members"]],
                          g["offsets"], stream=self.stream)

    # ---- passes --------------------------------------------------------------
    def forward(self):
        for i, L in enumerate(self.layers):
            epi = EPI_RELU if L.relu else EPI_NONE
            if L.kind == "conv":
                conv2d_fwd(fwd_desc(L), self.acts[i], self.w[i], self.acts[i + 1],
                           epi, ws=self.ws, stream=self.stream)
            else:
                conv_transpose2d_fwd(fwd_desc(L), self.acts[i], self.w[i],
                                     self.acts[i + 1], epi, ws=self.ws,
                                     stream=self.stream)
        return self.acts[-1]

    def head_grad(self, target):
        """g[L] = fp16(2*S*(y - t)/numel): loss-scaled MSE gradient."""
        y = self.acts[-1]
        l2_head_grad(y, target, 2.0 * self.loss_scale / y.numel(), self.g[-1],
                     stream=self.stream)

    def set_output_grad(self, dy):
        """Seed g[L] with a given gradient w.r.t. the chain output (after the
        last ReLU, if any: it is applied here)."""
        dy = torch.as_tensor(dy).to(self.dev).contiguous()
        if self.layers[-1].relu:
            relu_backward(dy, self.acts[-1], self.g[-1], stream=self.stream)
        else:
            self.g[-1].copy_(dy)

    def _bwd_weight(self, d, x, dy, i):
        if self.zero_copy and self.groups is not None:
            gi = self._group_of[i]
            conv2d_bwd_weight_checked(d, x, dy, self.dw[i], self.flags[gi:gi + 1],
                                      self.ws, stream=self.stream)
        else:
            conv2d_bwd_weight(d, x, dy, self.dw[i], self.ws, stream=self.stream)

    def backward(self, grad_path=False):
        if self.zero_copy and self.groups is not None:
            grad_flags_clear(self.flags, stream=self.stream)
        for i in reversed(range(len(self.layers))):
            L = self.layers[i]
            dy = self.g[i + 1]
            gate = i > 0 and self.layers[i - 1].relu
            epi = EPI_GATE if gate else EPI_NONE
            gt = self.acts[i] if gate else None
            if L.kind == "conv":
                d = fwd_desc(L)
                self._bwd_weight(d, self.acts[i], dy, i)
                conv2d_bwd_data(d, dy, self.w[i], self.g[i], epi, gt,
                                ws=self.ws, stream=self.stream)
            else:
                self._bwd_weight(convt_dw_desc(L), dy, self.acts[i], i)
                conv2d_fwd(convt_dx_desc(L), dy, self.w[i], self.g[i], epi, gt,
                           ws=self.ws, stream=self.stream)
            if grad_path and self.groups is not None and i in self._group_done_at:
                self.run_group(self._group_done_at[i])

    def observe(self):
        """Outcome of the last step a program ran: wait for its flag copy,
        then advance the loss scaler and the count of applied updates. A
        program does this by itself before each step's head call (the next
        forward pass is queued by then); call it after the last step to bring
        the host state up to date."""
        pend = getattr(self, "_pending", None)
        if pend is None:
            return
        self._pending = None
        ev, hf = pend
        ev.synchronize()
        found = bool(hf.any())
        self.last_found = found
        if self.scaler is not None:
            self.scaler.update(found)
            self.loss_scale = self.scaler.scale
        if not found and self.opt is not None:
            self.applied += 1

    def step(self, target):
        """Forward, loss head, backward, the grouped gradient path and, with
        an optimizer, the update."""
        if self.groups is not None:
            key = target.data_ptr()
            if getattr(self, "_prog_key", None) != key:
                self._prog = self.program(target)
                self._prog_key = key
            self._prog.run()
            self._prog.join()
            return
        self.forward()
        self.head_grad(target)
        self.backward()

    # ---- accounting -------------------------------------------------------------
    def conv_flops(self):
        """Algorithmic flops of one forward + backward pass (3 passes/layer)."""
        return sum(3 * L.flops for L in self.layers)

    # ---- prepared step -----------------------------------------------------------
    def program(self, target, streams=3, sync_every=1):
        """The step as a list of library calls with every argument marshalled
        once (descriptors, pointers, segment tables); running it costs one
        foreign call per launch. Same calls as ``step``; see StepProgram for
        the streams."""
        return StepProgram(self, target, streams, sync_every)


# algorithmic HBM bytes of the optimizer per parameter: w, m, v and the
# gradient read (12 + 4 for fp32 gradients, 12 + 2 for fp16 ones) and w, m,
# v and the fp16 copy written (14). The norms pass reads, the apply pass
# reads and writes.
OPT_READ_BYTES = 12
OPT_WRITE_BYTES = 14

# label, main kernel, algorithmic work (flops, or bytes for the gradient
# path), C function (None: a Python callable), argument tuple (the stream
# last), whether the call is exactly one launch of that kernel, its stream
# (0: main, 1: kernel gradients, 2: gradient path), the calls (indices)
# that must finish before it starts, and the later calls whose launch in the
# previous run must finish before it starts
Call = namedtuple("Call", "label kernel work fn args single sid deps prev_deps",
                  defaults=(True, 0, (), ()))


def kernel_gradient_workspace_bytes(layers):
    """Largest workspace of the chain's kernel-gradient passes."""
    ws = 0
    for L in layers:
        d = fwd_desc(L) if L.kind == "conv" else convt_dx_desc(L)
        ws = max(ws, workspace_bytes(d, OP_BWD_WEIGHT))
    return ws


class StepProgram:
    """The step as prepared library calls on up to three streams.

    The main stream runs the forward pass, the loss head and the
    input-gradient chain; stream 1 runs every kernel gradient as soon as its
    output gradient exists (an event recorded after the pass that wrote it);
    stream 2 runs each group's pack, unscale and unpack once the group's last
    kernel gradient is written. Kernel gradients and the gradient path thus
    fill the CUs that the input-gradient kernels leave idle (partial waves,
    tails) and the other way round. Stream 1 has its own workspace. The main
    stream waits for the other streams' last calls at the end of the step, so
    the next step's forward pass cannot overwrite activations a kernel
    gradient still reads, nor its kernel gradients a buffer a pack still
    reads. Every kernel is deterministic and reads only finished inputs, so
    the results are identical to the one-stream order (``streams=1``).

    With an optimizer, stream 2 also runs each group's optimizer norms pass
    (the part that reads the gradients; it writes only the workspace) right
    after the group's gradient path. With zero-copy groups the norms and
    updates read the fp16 loss-scaled gradients in the group slots, and the
    unscale and unpack are left out (the kernel gradients raise the flags).
    With an optimizer or a loss scaler, stream 2 then copies the group flags
    to pinned host memory; the next run waits for that copy just before its
    head call (its forward pass already queued), updates the scaler and the
    applied count, and patches the loss-scale and learning-rate arguments.
    The updates follow, one call per layer in forward order (layer 0's on
    stream 1, after the main stream's last pass, which reads its fp16
    weights). The main stream does not wait for them at the end of the
    run: the next run's forward pass of each layer waits for that layer's
    update, so the updates overlap the next forward pass. ``join()`` makes
    the main stream wait for everything."""

    def __init__(self, ch, target, streams=3, sync_every=1):
        if ch.groups is None:
            raise ValueError("the step program needs gradient groups")
        if streams not in (1, 3):
            raise ValueError("streams must be 1 or 3")
        L_ = lib()
        if ch.stream is not None:
            main = torch.cuda.ExternalStream(ch.stream, device=ch.dev)
        else:
            main = torch.cuda.current_stream(ch.dev)
        if streams == 3:  # default priorities
            self.streams = (main, torch.cuda.Stream(device=ch.dev),
                            torch.cuda.Stream(device=ch.dev))
        else:
            self.streams = (main,)
        sptr = [ctypes.c_void_p(x.cuda_stream) for x in self.streams]
        self._keep = [target]
        calls = []
        ws, wsb = ch.ws.data_ptr(), ch.ws.numel()
        ws_side = torch.empty(max(kernel_gradient_workspace_bytes(ch.layers), 16),
                              dtype=torch.uint8, device=ch.dev)
        self._keep.append(ws_side)
        ws2, wsb2 = ws_side.data_ptr(), ws_side.numel()
        nl = len(ch.layers)
        st = None  # placeholder: each call's stream is filled in below

        def ptr(t):
            return None if t is None else t.data_ptr()

        def desc(d):
            self._keep.append(d)
            return ctypes.byref(d)

        def one(d, op):  # no workspace: no split, one kernel launch
            return workspace_bytes(d, op) == 0

        for i, L in enumerate(ch.layers):
            epi = EPI_RELU if L.relu else EPI_NONE
            d = fwd_desc(L)
            if L.kind == "conv":
                calls.append(Call(f"{L.name}.fwd", kernel_name(d, OP_FWD), L.flops,
                                  L_.conv2d_fwd,
                                  (desc(d), ptr(ch.acts[i]), ptr(ch.w[i]),
                                   ptr(ch.acts[i + 1]), epi, None, ws, wsb, st),
                                  one(d, OP_FWD)))
            else:
                calls.append(Call(f"{L.name}.fwd", kernel_name(d, OP_CONVT), L.flops,
                                  L_.conv_transpose2d_fwd,
                                  (desc(d), ptr(ch.acts[i]), ptr(ch.w[i]),
                                   ptr(ch.acts[i + 1]), epi, None, ws, wsb, st),
                                  one(d, OP_CONVT)))
        y = ch.acts[-1]
        # loss-scale arguments, patched in place before each run
        self._ny = y.numel()
        self._head_scale = ctypes.c_double(2.0 * ch.loss_scale / self._ny)
        self._inv_scale = ctypes.c_float(1.0 / ch.loss_scale)
        calls.append(Call("head_grad", "head_grad_kernel", 6 * y.numel(),
                          L_.l2_head_grad,
                          (ptr(y), ptr(target), y.numel(), self._head_scale,
                           ptr(ch.g[-1]), st)))
        self._head = len(calls) - 1
        writer = {nl: len(calls) - 1}  # call that writes g[i]
        # the non-finite flags are raised by the unscale calls (stream 2) and,
        # with zero-copy groups, by the kernel gradients (stream 1); cleared
        # after the head call, which follows the previous step's last reads
        calls.append(Call("flags.clear", "flags_clear_kernel", 0, L_.grad_flags_clear,
                          (ch.flags.data_ptr(), ch.flags.numel(), st), True,
                          sid=1 if ch.zero_copy else 2, deps=(self._head,)))
        zc = ch.zero_copy

        def dw_call(label, kname, flops, d, x, dy, i):
            if zc:
                gi = ch._group_of[i]
                flag = ch.flags[gi:gi + 1]
                self._keep.append(flag)
                return Call(label, kname, flops, L_.conv2d_bwd_weight_checked,
                            (desc(d), ptr(x), ptr(dy), ptr(ch.dw[i]), flag.data_ptr(),
                             ws2, wsb2, st), one(d, OP_BWD_WEIGHT),
                            sid=1, deps=(writer[i + 1],))
            return Call(label, kname, flops, L_.conv2d_bwd_weight,
                        (desc(d), ptr(x), ptr(dy), ptr(ch.dw[i]), ws2, wsb2, st),
                        one(d, OP_BWD_WEIGHT), sid=1, deps=(writer[i + 1],))
        self.params = None
        if ch.opt is not None:
            # with zero-copy groups the optimizer reads each layer's fp16
            # loss-scaled gradient in its group slot (flags come from the
            # kernel gradients, so no unscale or unpack is needed); otherwise
            # the fp32 gradients the unpack writes
            o = ch.opt
            self.params = OptParams(o.lr_at(ch.applied), o.beta1, o.beta2, o.eps,
                                    o.weight_decay)
            fused = ch.zero_copy
            tab = opt_tensors(ch.w32, ch.w, ch.m, ch.v, ch.dw) if fused else ch.opt_tensors
            self._opt = dict(tab=tab, fmt=GRAD_F16_SCALED if fused else GRAD_F32,
                             inv=self._inv_scale if fused else ctypes.c_float(1.0),
                             gb=2 if fused else 4, h="true" if fused else "false",
                             fused=fused, n=sum(w.numel() for w in ch.w32))
            self._keep.append(tab)
        last_dw = {}

        def emit_dw(j, dep):
            """Kernel gradient of layer j (after the call `dep` that wrote
            g[j + 1] or a later input gradient), then its group's path if j
            completes a group."""
            L = ch.layers[j]
            if L.kind == "conv":
                d = fwd_desc(L)
                c = dw_call(f"{L.name}.dW", kernel_name(d, OP_BWD_WEIGHT), L.flops, d,
                            ch.acts[j], ch.g[j + 1], j)
            else:
                d = convt_dx_desc(L)
                c = dw_call(f"{L.name}.dW", kernel_name(d, OP_BWD_WEIGHT), L.flops, d,
                            ch.g[j + 1], ch.acts[j], j)
            calls.append(c._replace(deps=(dep,)))
            last_dw[j] = len(calls) - 1
            gi = ch._group_done_at.get(j)
            if gi is not None:
                gc = self._group_calls(ch, gi, L_, st) + self._norms_calls(ch, gi, L_, st)
                gc[0] = gc[0]._replace(deps=(last_dw[j],))
                calls.extend(gc)

        # kernel gradients are issued sync_every layers at a time, all after
        # the latest input gradient: the main stream then records one event
        # per sync_every layers for the kernel-gradient stream to wait on
        pending = []
        for i in reversed(range(nl)):
            L = ch.layers[i]
            dy = ch.g[i + 1]
            gate = i > 0 and ch.layers[i - 1].relu
            epi = EPI_GATE if gate else EPI_NONE
            gt = ptr(ch.acts[i]) if gate else None
            pending.append(i)
            if len(pending) >= sync_every or i == 0:
                for j in pending:
                    emit_dw(j, writer[i + 1])
                pending = []
            if L.kind == "conv":
                d = fwd_desc(L)
                calls.append(Call(f"{L.name}.dx", kernel_name(d, OP_BWD_DATA),
                                  L.flops, L_.conv2d_bwd_data,
                                  (desc(d), ptr(dy), ptr(ch.w[i]), ptr(ch.g[i]), epi,
                                   gt, ws, wsb, st), one(d, OP_BWD_DATA)))
            else:
                d = convt_dx_desc(L)
                calls.append(Call(f"{L.name}.dx", kernel_name(d, OP_FWD), L.flops,
                                  L_.conv2d_fwd,
                                  (desc(d), ptr(dy), ptr(ch.w[i]), ptr(ch.g[i]), epi,
                                   gt, ws, wsb, st), one(d, OP_FWD)))
            writer[i] = len(calls) - 1
        self._copy = None
        if ch.opt is not None or ch.scaler is not None:
            # the step's flags to pinned host memory once every flag is final
            # (after the last kernel gradient and unscale); read before the
            # next step's head call, by which time its forward pass is queued
            self.host_flags = torch.zeros(len(ch.groups), dtype=torch.int32,
                                          pin_memory=True)
            calls.append(Call("flags.copy", "", 0, None,
                              (lambda: self.host_flags.copy_(ch.flags,
                                                             non_blocking=True),),
                              False, sid=2))
            self._copy = len(calls) - 1
        self._apply = {}
        if ch.opt is not None:
            # each layer's update after every group's norms, in forward order
            # (the first apply call also forms tau): layers 1.. on stream 2,
            # layer 0 on stream 1 once the main stream's last pass (layer 0's
            # input gradient, which reads its fp16 weights) is done. The next
            # run's forward pass of layer i waits for the apply of layer i
            # only, so the updates overlap the next forward pass.
            o = self._opt
            order = [(i, 2) for i in range(1, nl)] + [(0, 1 if nl > 1 else 2)]
            for i, sid in order:
                deps = () if i else (writer[0],) + \
                    ((self._apply[1],) if nl > 1 else ())
                n_i = ch.w32[i].numel()
                calls.append(Call(f"{ch.layers[i].name}.apply",
                                  f"lars_adam_apply_kernel<{o['h']}>",
                                  (OPT_READ_BYTES + o["gb"] + OPT_WRITE_BYTES) * n_i,
                                  L_.lars_adam_apply,
                                  (o["tab"], nl, i, 1, ctypes.byref(self.params), o["fmt"],
                                   o["inv"], ch.flags.data_ptr(), len(ch.groups),
                                   ch.step_count.data_ptr(), ch.opt_ws.data_ptr(),
                                   ch.opt_ws.numel(), st), i != order[0][0], sid=sid,
                                  deps=deps))
                self._apply[i] = len(calls) - 1
            fwd = {f"{L.name}.fwd": i for i, L in enumerate(ch.layers)}
            calls = [c._replace(prev_deps=(self._apply[fwd[c.label]],))
                     if c.label in fwd else c for c in calls]
        if streams == 1:  # program order already respects every dependency
            calls = [c._replace(sid=0, deps=(), prev_deps=()) for c in calls]
        # the stream argument of each library call
        calls = [c if c.fn is None else
                 c._replace(args=c.args[:-1] + (sptr[c.sid],)) for c in calls]
        self.final = tuple(max(j for j, c in enumerate(calls) if c.sid == sid)
                           for sid in range(1, len(self.streams)))
        # what the main stream waits for at the end of a run: every side
        # stream's last call, except the per-layer updates on stream 2, which
        # the next run's forward pass waits for layer by layer (join() waits
        # for everything)
        self.step_final = tuple(j for j in self.final
                                if not (self._apply and calls[j].sid == 2))
        needed = {d for c in calls for d in c.deps + c.prev_deps} | set(self.final)
        if self._copy is not None:
            needed.add(self._copy)
        self.events = {j: torch.cuda.Event() for j in sorted(needed)}
        self.calls = calls
        self.ch = ch

    def _norms_calls(self, ch, gi, L_, st):
        if ch.opt is None:
            return []
        mem = sorted(ch.groups[gi]["members"])
        first, count = mem[0], len(mem)
        assert mem == list(range(first, first + count)), "a group is a layer range"
        o = self._opt
        n = sum(ch.w32[i].numel() for i in mem)
        return [Call(f"G{gi}.norms", f"lars_adam_norms_kernel<{o['h']}>",
                     (OPT_READ_BYTES + o["gb"]) * n, L_.lars_adam_norms,
                     (o["tab"], len(ch.layers), first, count, ctypes.byref(self.params),
                      o["fmt"], o["inv"], ch.step_count.data_ptr(), ch.opt_ws.data_ptr(),
                      ch.opt_ws.numel(), st), sid=2)]

    def _group_calls(self, ch, gi, L_, st):
        if ch.opt is not None and self._opt["fused"]:
            return []
        g = ch.groups[gi]
        n = g["numel"]
        src = (Segment * len(g["members"]))(
            *[Segment(ch.dw[m].data_ptr(), ch.dw[m].numel(), off)
              for m, off in zip(g["members"], g["offsets"])])
        dst = (Segment * len(g["members"]))(
            *[Segment(ch.master[m].data_ptr(), ch.master[m].numel(), off)
              for m, off in zip(g["members"], g["offsets"])])
        self._keep += [src, dst]
        g16, g32 = ch.gbuf16[gi], ch.gbuf32[gi]
        flag = ch.flags[gi:gi + 1]
        self._keep.append(flag)
        pack = [] if ch.zero_copy else [
            Call(f"G{gi}.pack", "copy_pieces_kernel<2>", 4 * n, L_.grad_group_pack,
                 (src, len(g["members"]), g16.data_ptr(), n, st), sid=2)]
        return pack + [
            Call(f"G{gi}.unscale", "unscale_vec_kernel", 6 * n, L_.grad_unscale_check,
                 (g16.data_ptr(), n, self._inv_scale, g32.data_ptr(),
                  flag.data_ptr(), st), sid=2),
            Call(f"G{gi}.unpack", "copy_pieces_kernel<4>", 8 * n, L_.grad_group_unpack,
                 (g32.data_ptr(), n, dst, len(g["members"]), st), sid=2),
        ]

    def _patch(self):
        ch = self.ch
        self._head_scale.value = 2.0 * ch.loss_scale / self._ny
        self._inv_scale.value = 1.0 / ch.loss_scale
        if self.params is not None:
            self.params.lr = ch.opt.lr_at(ch.applied)

    def run(self, events=None, kernel_events=None):
        """Run the step once. events: {call index: (start, end)} HIP events
        recorded around those calls on the call's stream; kernel_events: the
        same for convolution calls, recorded by the library around the call's
        main kernel only (fg_profile_next_launch)."""
        streams, evs = self.streams, self.events
        for i, c in enumerate(self.calls):
            if i == self._head:
                self.ch.observe()
                self._patch()
            s = streams[c.sid]
            for d in c.deps + c.prev_deps:
                s.wait_event(evs[d])
            ev = events.get(i) if events else None
            if ev:
                ev[0].record(s)
            kev = kernel_events.get(i) if kernel_events else None
            if kev:
                profile_next_launch(*kev)
            if c.fn is None:
                with torch.cuda.stream(s):
                    c.args[0]()
            else:
                st = c.fn(*c.args)
                if st:
                    raise FgError(c.label, st)
            if ev:
                ev[1].record(s)
            if i in evs:
                evs[i].record(s)
        for j in self.step_final:
            streams[0].wait_event(evs[j])
        if self._copy is not None:
            self.ch._pending = (evs[self._copy], self.host_flags)

    def join(self):
        """Make the main stream wait for all of the last run's work (the
        per-layer updates included)."""
        for j in self.final:
            self.streams[0].wait_event(self.events[j])
