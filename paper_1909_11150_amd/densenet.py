"""One GPU's share of a training step of the FC-DenseNet variant.

Section 6.2 (Neural Network Architecture) describes the paper's model as
an FC-DenseNet with growth rate 256 and average pooling; its loss (Model
Implementation) is the Huber loss. ``DenseNet`` runs the forward pass, the
loss-scaled Huber head gradient and the backward pass of such a network
(layer table from ``synth.densenet_layers``: stem, dense blocks on a down
path with transition-down 1x1 convs and 2x2 average pooling, a bottleneck
block, transposed-conv transitions up with skip concatenations, a 1x1 head)
entirely through libfcngrad calls, prepared once as a call list like the
chain's step program.

Dense concatenation. The convolutions read a channel prefix of a wider
buffer and write, or add, into a channel slice of one (pixel strides):
  * forward: each level d keeps one buffer laid out as [transition-up
    output | the down block's input and layer outputs (the skip) | the up
    block's layer outputs], the bottleneck one as [pooled input | layer
    outputs]. A layer reads the channels before its own slice and writes
    its slice, so every concatenation is in place; the stem writes the first
    down block's input slice, and a pooled map is copied into the next
    block's input slice. The last layer of a bottleneck or up block writes
    into the block's new-feature buffer, to which the other layers' outputs
    are copied (a transition up reads it dense);
  * backward: a bottleneck or up block keeps a gradient buffer G in the
    layout of its last concatenation. A layer's output gradient is its slice
    of G (of the new-feature gradient, for the last layer), gated by its ReLU
    output; its input gradient is added into the slices it read by the
    convolution itself (the accumulate epilogue). A down block's G is the
    skip's slice of its up block's G (a strided view), so the skip gradient
    is in place when the transition conv adds its input gradient to it.
fp16 storage throughout; every addition is one rounding.
"""
import ctypes
from collections import namedtuple

import torch

from . import (EPI_ACC, EPI_NONE, EPI_RELU, OP_BWD_DATA, OP_BWD_WEIGHT, OP_CONVT,
               OP_FWD, ConvDesc, FgError, Segment, grad_group_plan, kernel_name, lib,
               profile_next_launch, workspace_bytes)
from .fcn import (Call, chain_workspace_bytes, kernel_gradient_workspace_bytes)

F16 = torch.float16

# a channel slice of a buffer: base tensor, element offset of the first
# channel, pixel stride, channels
Slice = namedtuple("Slice", "t off ld ch")


def _dense(t):
    return Slice(t, 0, t.shape[-1], t.shape[-1])


def _structure(layers):
    names = [L.name for L in layers]
    levels = sum(1 for n in names if n.startswith("TD"))
    per = sum(1 for n in names if n.startswith("B."))
    for req in ["C0", "F1x1"] + [f"TD{d}" for d in range(1, levels + 1)] + \
               [f"TU{d}" for d in range(1, levels + 1)]:
        if req not in names:
            raise ValueError(f"layer {req} missing from the dense network")
    return levels, per


def _desc(L, op, x_ld=0, y_ld=0):
    """Descriptor of one pass; for a transposed conv's input gradient and
    kernel gradient, the conv of dy (the big image) with Wt read as KRSC."""
    n, h, w, c = L.x_shape
    if L.kind == "conv" or op == OP_CONVT:
        return ConvDesc.make(n, h, w, c, L.y_shape[3], L.r, L.s, L.stride, L.pad,
                             x_ld, y_ld)
    n, ho, wo, co = L.y_shape
    return ConvDesc.make(n, ho, wo, co, c, L.r, L.s, L.stride, L.pad, x_ld, y_ld)


class DenseNet:
    def __init__(self, layers, weights, x, loss_scale=2.0 ** 15, delta=10.0,
                 device="cuda", stream=None, group_cap_bytes=None, group_align_bytes=256):
        self.layers = list(layers)
        self.L = {L.name: L for L in self.layers}
        self.levels, self.per = _structure(self.layers)
        self.k = self.L["D1.1"].y_shape[3]
        self.dev = torch.device(device)
        self.stream = stream
        self.loss_scale, self.delta = float(loss_scale), float(delta)
        e = lambda s: torch.empty(s, dtype=F16, device=self.dev)
        self.x = torch.as_tensor(x).to(self.dev).contiguous()
        self.w = {L.name: torch.as_tensor(w).to(self.dev).contiguous()
                  for L, w in zip(self.layers, weights)}
        self.dw = {L.name: e(L.w_shape) for L in self.layers}
        self.ws = torch.empty(max(chain_workspace_bytes(self.layers), 16),
                              dtype=torch.uint8, device=self.dev)
        # forward buffers: one per level (Z["U<d>"]) and the bottleneck's
        # (Z["B"]), pooled maps, new-feature buffers; where each layer reads
        # its input (inp) and writes its (post-ReLU) output (out)
        self.Z, self.P, self.NF, self.G, self.dNF = {}, {}, {}, {}, {}
        self.inp, self.out = {}, {}
        k, per = self.k, self.per
        nk = per * k
        for d in range(1, self.levels + 1):
            n_, h, w, c0u = self.L[f"U{d}.1"].x_shape
            c0d = self.L[f"D{d}.1"].x_shape[3]
            z = e((n_, h, w, c0u + (per - 1) * k))
            self.Z[f"U{d}"] = z
            ld = z.shape[3]
            for l in range(1, per + 1):
                self.inp[f"D{d}.{l}"] = Slice(z, nk, ld, c0d + (l - 1) * k)
                self.out[f"D{d}.{l}"] = Slice(z, nk + c0d + (l - 1) * k, ld, k)
            self.inp[f"TD{d}"] = Slice(z, nk, ld, c0d + per * k)     # the skip
            self.out[f"TU{d}"] = Slice(z, 0, ld, nk)
            self._block_tail(f"U{d}", z, c0u)
            tdy = self.L[f"TD{d}"].y_shape
            self.out[f"TD{d}"] = _dense(e(tdy))
            self.P[d] = e((tdy[0], tdy[1] // 2, tdy[2] // 2, tdy[3]))
        n_, h, w, c0b = self.L["B.1"].x_shape
        self.Z["B"] = e((n_, h, w, c0b + (per - 1) * k))
        self._block_tail("B", self.Z["B"], c0b)
        self.out["C0"] = self.inp["D1.1"]._replace(ch=self.L["C0"].y_shape[3])
        self.out["F1x1"] = _dense(e(self.L["F1x1"].y_shape))
        # post-ReLU outputs as (possibly strided) tensor views
        self.act = {name: self._view(s) for name, s in self.out.items()}
        # gradients: one output-gradient buffer per layer (its kernel
        # gradient may still read it on the side stream)
        self.g_out = e(self.L["F1x1"].y_shape)
        self.dX = e(self.x.shape)
        self.dY = {f"{b}.{l}": e(self.L[f"{b}.{l}"].y_shape)
                   for b in self._blocks() for l in range(1, self.per + 1)}
        self.dT = {d: e(self.L[f"TD{d}"].y_shape) for d in range(1, self.levels + 1)}
        self.dP = {d: e(self.P[d].shape) for d in range(1, self.levels + 1)}
        self.dU = {d: e(self.L[f"TU{d}"].y_shape) for d in range(1, self.levels + 1)}
        self.dC0 = e(self.L["C0"].y_shape)
        self.groups = None
        if group_cap_bytes is not None:
            self._plan_groups(group_cap_bytes, group_align_bytes)
        self._L = lib()

    def dw_order(self):
        """Layer names in the order the backward pass completes their kernel
        gradients: head, up levels from the top, bottleneck, down levels from
        the bottom, stem; within a block, its last layer first."""
        blk = lambda b: [f"{b}.{l}" for l in range(self.per, 0, -1)]
        order = ["F1x1"]
        for d in range(1, self.levels + 1):
            order += blk(f"U{d}") + [f"TU{d}"]
        order += blk("B")
        for d in range(self.levels, 0, -1):
            order += [f"TD{d}"] + blk(f"D{d}")
        return order + ["C0"]

    def _plan_groups(self, cap, align):
        """Gradient groups (Section 4.2) over the kernel gradients in
        completion order, as the chain forms them: fp16 group buffers, their
        fp32 unscaled copies, a non-finite flag per group and fp32 master
        gradients per layer."""
        order = self.dw_order()
        gof, oof, gnum = grad_group_plan([self.dw[m].numel() for m in order], cap,
                                         align, 2)
        self.groups = [{"members": [order[j] for j in range(len(order)) if gof[j] == g],
                        "offsets": [oof[j] for j in range(len(order)) if gof[j] == g],
                        "numel": n} for g, n in enumerate(gnum)]
        e = lambda n, dt: torch.empty(n, dtype=dt, device=self.dev)
        self.gbuf16 = [e(g["numel"], F16) for g in self.groups]
        self.gbuf32 = [e(g["numel"], torch.float32) for g in self.groups]
        self.flags = torch.zeros(len(self.groups), dtype=torch.int32, device=self.dev)
        self.master = {L.name: e(L.w_shape, torch.float32) for L in self.layers}
        self._group_done_at = {g["members"][-1]: gi for gi, g in enumerate(self.groups)}

    @staticmethod
    def _view(s):
        n, h, w = s.t.shape[:3]
        return s.t.view(n, h, w, s.ld)[..., s.off:s.off + s.ch]

    def _blocks(self):
        return [f"D{d}" for d in range(1, self.levels + 1)] + ["B"] + \
               [f"U{d}" for d in range(1, self.levels + 1)]

    def _block_tail(self, blk, z, c0):
        """Slices of a bottleneck or up block whose input is the first c0
        channels of z, its new-feature and gradient buffers."""
        e = lambda s: torch.empty(s, dtype=F16, device=self.dev)
        n, h, w = z.shape[:3]
        k, per, ld = self.k, self.per, z.shape[3]
        self.NF[blk] = e((n, h, w, per * k))
        self.dNF[blk] = e((n, h, w, per * k))
        self.G[blk] = e((n, h, w, c0 + per * k))
        for l in range(1, per + 1):
            self.inp[f"{blk}.{l}"] = Slice(z, 0, ld, c0 + (l - 1) * k)
            self.out[f"{blk}.{l}"] = Slice(z, c0 + (l - 1) * k, ld, k) if l < per else \
                Slice(self.NF[blk], (l - 1) * k, per * k, k)

    # ---- prepared calls ----------------------------------------------------------
    def program(self, target, streams=2):
        """streams = 1: every call in order on one stream; 2: the kernel
        gradients on a second stream; 3: also the forward pass's copies into
        the new-feature buffers on a third."""
        if streams < 1:
            raise ValueError("streams must be >= 1")
        return _DenseProgram(self, target, min(streams, 3))

    def step(self, target):
        key = target.data_ptr()
        if getattr(self, "_prog_key", None) != key:
            self._prog = self.program(target)
            self._prog_key = key
        self._prog.run()
        self._prog.join()

    def conv_flops(self):
        return sum(3 * L.flops for L in self.layers)


class _DenseProgram:
    """The step as a list of prepared library calls (the chain step
    program's interface: calls, streams, events, run, join). With two
    streams each kernel gradient runs on the second one as soon as its
    output gradient is written (an event after the writing call), beside the
    main stream's input gradients and copies, with a workspace of its own.
    With three, the forward pass's copies into the new-feature buffers,
    which no later layer of the block waits for, run on the third, each
    after the layer it copies. The main stream waits for
    the other streams' last calls at the end of the step, before the next
    forward pass overwrites what they read. Every kernel reads only
    finished inputs, so the results equal the one-stream order's."""

    def __init__(self, net, target, streams=1):
        self.net = net
        self._keep = [target]
        self.calls = []
        self._L = lib()
        main = torch.cuda.ExternalStream(net.stream, device=net.dev) \
            if net.stream is not None else torch.cuda.current_stream(net.dev)
        self.streams = (main,) + tuple(torch.cuda.Stream(device=net.dev)
                                       for _ in range(streams - 1))
        self._dw_sid = 1 if streams > 1 else 0
        self._cp_sid = 2 if streams > 2 else 0
        self._sp = [ctypes.c_void_p(x.cuda_stream) for x in self.streams]
        self._dw_seen = []
        self._ws_side = torch.empty(
            max(16, kernel_gradient_workspace_bytes(net.layers)), dtype=torch.uint8,
            device=net.dev) if streams > 1 else net.ws
        self._build(target)
        if streams == 1:
            self.calls = [c._replace(sid=0, deps=()) for c in self.calls]
        # a dependency on a call of the same stream is its stream order
        self.calls = [c._replace(deps=tuple(d for d in c.deps if self.calls[d].sid != c.sid))
                      for c in self.calls]
        self.calls = [c if c.fn is None else c._replace(args=c.args + (self._sp[c.sid],))
                      for c in self.calls]
        self.final = tuple(max(j for j, c in enumerate(self.calls) if c.sid == sid)
                           for sid in range(1, len(self.streams)))
        self.step_final = self.final
        needed = {d for c in self.calls for d in c.deps} | set(self.final)
        self.events = {j: torch.cuda.Event() for j in sorted(needed)}

    # -- checks: every buffer a call touches holds what the call addresses --
    @staticmethod
    def _span_ok(s, npix):
        need = s.off + (npix - 1) * s.ld + s.ch
        if s.t.dtype != F16 or not s.t.is_contiguous() or s.t.numel() < need or \
                s.ch > s.ld:
            raise ValueError(f"buffer of {s.t.numel()} fp16 elements, call reaches {need}")

    @staticmethod
    def _shape_ok(t, shape):
        if tuple(t.shape) != tuple(shape) or not t.is_contiguous():
            raise ValueError(f"tensor {tuple(t.shape)} where {tuple(shape)} is needed")

    def _keep_desc(self, d):
        self._keep.append(d)
        return ctypes.byref(d)

    def _add(self, label, kernel, work, fn, args, single=True, sid=0, deps=()):
        """Append a call; the stream argument is added once all are built."""
        self.calls.append(Call(label, kernel, work, fn, args, single, sid, deps))
        return len(self.calls) - 1

    @staticmethod
    def _ptr(s):
        return s.t.data_ptr() + 2 * s.off

    # -- ops --
    def _in_ok(self, x, L):
        """x: the slice a layer reads as its input (L.x_shape)."""
        assert x.ch == L.x_shape[3]
        self._span_ok(x, L.x_shape[0] * L.x_shape[1] * L.x_shape[2])

    def conv_fwd(self, name, x, out, relu, deps=()):
        """Forward pass of a layer: input from slice x (dense for a
        transposed conv), output into slice out."""
        L = self.net.L[name]
        n = self.net
        self._in_ok(x, L)
        npix = L.y_shape[0] * L.y_shape[1] * L.y_shape[2]
        assert out.ch == L.y_shape[3]
        self._span_ok(out, npix)
        op = OP_FWD if L.kind == "conv" else OP_CONVT
        if op == OP_CONVT:
            assert x.ld == x.ch
        d = _desc(L, op, x_ld=x.ld, y_ld=out.ld)
        fn = self._L.conv2d_fwd if L.kind == "conv" else self._L.conv_transpose2d_fwd
        return self._add(f"{name}.fwd", kernel_name(d, op), L.flops, fn,
                         (self._keep_desc(d), self._ptr(x), n.w[name].data_ptr(),
                          self._ptr(out), EPI_RELU if relu else EPI_NONE, None,
                          n.ws.data_ptr(), n.ws.numel()), workspace_bytes(d, op) == 0,
                         deps=deps)

    def conv_bwd(self, name, x, dy, dx, acc):
        """Kernel gradient into dw[name] (second stream, after the call that
        wrote dy, which is the last one appended); input gradient into slice
        dx, added to what it holds when acc (no gate)."""
        L = self.net.L[name]
        n = self.net
        self._in_ok(x, L)
        self._shape_ok(dy, L.y_shape)
        npix = L.x_shape[0] * L.x_shape[1] * L.x_shape[2]
        assert dx.ch == L.x_shape[3]
        self._span_ok(dx, npix)
        wsp, wsb = n.ws.data_ptr(), n.ws.numel()
        dws, dwb = self._ws_side.data_ptr(), self._ws_side.numel()
        epi = EPI_ACC if acc else EPI_NONE
        dwk = dict(sid=self._dw_sid, deps=(len(self.calls) - 1,))
        if L.kind == "conv":
            d = _desc(L, OP_FWD, x_ld=dx.ld)
            dw_d = _desc(L, OP_FWD, x_ld=x.ld)
            self._add(f"{name}.dW", kernel_name(dw_d, OP_BWD_WEIGHT), L.flops,
                      self._L.conv2d_bwd_weight,
                      (self._keep_desc(dw_d), self._ptr(x), dy.data_ptr(),
                       n.dw[name].data_ptr(), dws, dwb),
                      workspace_bytes(dw_d, OP_BWD_WEIGHT) == 0, **dwk)
            self._add(f"{name}.dx", kernel_name(d, OP_BWD_DATA), L.flops,
                      self._L.conv2d_bwd_data,
                      (self._keep_desc(d), dy.data_ptr(), n.w[name].data_ptr(),
                       self._ptr(dx), epi, None, wsp, wsb),
                      workspace_bytes(d, OP_BWD_DATA) == 0)
        else:   # transposed conv: both passes are convs of dy with Wt as KRSC
            assert x.ld == x.ch
            dw_d = _desc(L, OP_BWD_WEIGHT)
            self._add(f"{name}.dW", kernel_name(dw_d, OP_BWD_WEIGHT), L.flops,
                      self._L.conv2d_bwd_weight,
                      (self._keep_desc(dw_d), dy.data_ptr(), self._ptr(x),
                       n.dw[name].data_ptr(), dws, dwb),
                      workspace_bytes(dw_d, OP_BWD_WEIGHT) == 0, **dwk)
            d = _desc(L, OP_BWD_DATA, y_ld=dx.ld)
            self._add(f"{name}.dx", kernel_name(d, OP_FWD), L.flops, self._L.conv2d_fwd,
                      (self._keep_desc(d), dy.data_ptr(), n.w[name].data_ptr(),
                       self._ptr(dx), epi, None, wsp, wsb),
                      workspace_bytes(d, OP_FWD) == 0)
        self._dw_seen.append(name)
        if n.groups is not None and name in n._group_done_at:
            self._group_calls(n._group_done_at[name])

    def _group_calls(self, gi):
        """Pack, unscale with the non-finite check, unpack (Sections 4.2 and
        6.2) of a group once its last kernel gradient is written: on the
        kernel-gradient stream, after every member's kernel gradient."""
        n = self.net
        g = n.groups[gi]
        num = g["numel"]
        seg = lambda ts: (Segment * len(ts))(
            *[Segment(t.data_ptr(), t.numel(), off) for t, off in zip(ts, g["offsets"])])
        src = seg([n.dw[m] for m in g["members"]])
        dst = seg([n.master[m] for m in g["members"]])
        flag = n.flags[gi:gi + 1]
        self._keep += [src, dst, flag]
        g16, g32 = n.gbuf16[gi], n.gbuf32[gi]
        sid = self._dw_sid
        self._add(f"G{gi}.pack", "copy_pieces_kernel<2>", 4 * num, self._L.grad_group_pack,
                  (src, len(g["members"]), g16.data_ptr(), num), sid=sid)
        self._add(f"G{gi}.unscale", "unscale_vec_kernel", 6 * num,
                  self._L.grad_unscale_check,
                  (g16.data_ptr(), num, self._inv_scale, g32.data_ptr(), flag.data_ptr()),
                  sid=sid)
        self._add(f"G{gi}.unpack", "copy_pieces_kernel<4>", 8 * num,
                  self._L.grad_group_unpack,
                  (g32.data_ptr(), num, dst, len(g["members"])), sid=sid)

    def copy(self, label, src, dst, gate=None, acc=False, sid=0, deps=()):
        """Per pixel, dst.ch channels from slice src to slice dst (gated by
        slice gate; added to dst when acc)."""
        npix = dst.t.numel() // dst.ld
        nch = dst.ch
        for s in (src, dst) + ((gate,) if gate is not None else ()):
            assert s.ch == nch
            self._span_ok(s, npix)
        rd = 2 * nch * npix * (2 if acc else 1) + (2 * nch * npix if gate is not None else 0)
        return self._add(label, f"channel_slice_copy_kernel<{'true' if acc else 'false'}>",
                         rd + 2 * nch * npix, self._L.channel_slice_copy,
                         (self._ptr(src), src.ld,
                          None if gate is None else self._ptr(gate),
                          0 if gate is None else gate.ld,
                          self._ptr(dst), dst.ld, npix, nch, int(acc)),
                         sid=sid, deps=deps)

    # -- the step --
    def _block_fwd(self, blk, ready):
        """Dense layers of a block whose input slice is complete once the
        calls in `ready` are. Each layer reads the channels before its own
        slice and writes its slice. Returns the calls that complete the
        block's outputs: its last layer (down blocks; the skip is then
        whole) or the new-feature buffer (others)."""
        n = self.net
        nf_ready = []
        for l in range(1, n.per + 1):
            name = f"{blk}.{l}"
            conv = self.conv_fwd(name, n.inp[name], n.out[name], True, deps=ready)
            ready = (conv,)
            if blk.startswith("D"):
                continue
            if l < n.per:     # copied into the new-feature buffer
                nf = n.NF[blk]
                nf_ready.append(self.copy(f"{name}.new", n.out[name],
                                          Slice(nf, (l - 1) * n.k, nf.shape[3], n.k),
                                          sid=self._cp_sid, deps=(conv,)))
            else:
                nf_ready.append(conv)
        return ready if blk.startswith("D") else tuple(nf_ready)

    def _block_bwd(self, blk, G, c0, fresh, dnf=None):
        """G: slice over the layout of the block's last concatenation (ld =
        its pixel stride). For a fresh block (bottleneck, up) nothing is in G
        yet and dnf holds the new-feature gradient; otherwise G holds the
        whole gradient. Leaves the block input's gradient in G's first c0
        channels."""
        n = self.net
        nk = n.per * n.k
        for l in range(n.per, 0, -1):
            name = f"{blk}.{l}"
            lo = c0 + (l - 1) * n.k
            dY = n.dY[name]
            src = Slice(dnf, (l - 1) * n.k, nk, n.k) if fresh and l == n.per else \
                Slice(G.t, G.off + lo, G.ld, n.k)
            self.copy(f"{name}.dy", src, _dense(dY), gate=n.out[name])
            first = fresh and l == n.per          # nothing in G to add to yet
            self.conv_bwd(name, n.inp[name], dY, Slice(G.t, G.off, G.ld, lo),
                          acc=not first)
            if first and n.per > 1:   # the earlier layers' new-feature gradients
                self.copy(f"{blk}.dnew", Slice(dnf, 0, nk, lo - c0),
                          Slice(G.t, G.off + c0, G.ld, lo - c0), acc=True)

    def _build(self, target):
        n = self.net
        Lb = self._L
        nk = n.per * n.k
        self._inv_scale = ctypes.c_float(1.0 / n.loss_scale)
        if n.groups is not None:     # the step's non-finite flags start clear
            self._add("flags.clear", "flags_clear_kernel", 0, Lb.grad_flags_clear,
                      (n.flags.data_ptr(), n.flags.numel()), sid=self._dw_sid)
        # ---- forward
        self.conv_fwd("C0", _dense(n.x), n.out["C0"], True)
        ready = (len(self.calls) - 1,)
        skip_ready = {}
        for d in range(1, n.levels + 1):
            skip_ready[d] = self._block_fwd(f"D{d}", ready)
            self.conv_fwd(f"TD{d}", n.inp[f"TD{d}"], n.out[f"TD{d}"], True,
                          deps=skip_ready[d])
            td = n.act[f"TD{d}"]
            self._add(f"TD{d}.pool", "avg_pool2d_fwd_kernel", 2 * td.numel() * 5 // 4,
                      Lb.avg_pool2d_fwd,
                      (td.data_ptr(), *td.shape, n.P[d].data_ptr()))
            # the pooled map into the next block's input slice
            nxt = n.inp[f"D{d + 1}.1" if d < n.levels else "B.1"]
            ready = (self.copy(f"P{d}.cat", _dense(n.P[d]), nxt),)
        nf_ready = self._block_fwd("B", ready)
        nf = n.NF["B"]
        tu_in = {}
        for d in range(n.levels, 0, -1):
            tu = f"TU{d}"
            tu_in[d] = nf
            tconv = self.conv_fwd(tu, _dense(nf), n.out[tu], True, deps=nf_ready)
            nf_ready = self._block_fwd(f"U{d}", (tconv,) + tuple(skip_ready[d]))
            nf = n.NF[f"U{d}"]
        y = n.act["F1x1"]
        self.conv_fwd("F1x1", _dense(nf), n.out["F1x1"], False, deps=nf_ready)
        # ---- head: loss-scaled mean Huber loss
        self._head_args = [y.data_ptr(), target.data_ptr(), y.numel(),
                           ctypes.c_double(n.loss_scale / y.numel()),
                           ctypes.c_double(n.delta), n.g_out.data_ptr()]
        self._add("head_grad", "huber_head_grad_kernel", 10 * y.numel(),
                  Lb.huber_head_grad, tuple(self._head_args))
        # ---- backward: head, up blocks (level 1 first), bottleneck, down path
        self.conv_bwd("F1x1", _dense(nf), n.g_out, _dense(n.dNF["U1"]), acc=False)
        for d in range(1, n.levels + 1):
            blk, tu = f"U{d}", f"TU{d}"
            G = _dense(n.G[blk])
            self._block_bwd(blk, G, n.inp[f"{blk}.1"].ch, True, n.dNF[blk])
            self.copy(f"{tu}.dy", Slice(G.t, 0, G.ld, nk), _dense(n.dU[d]),
                      gate=n.out[tu])
            below = "B" if d == n.levels else f"U{d + 1}"
            self.conv_bwd(tu, _dense(tu_in[d]), n.dU[d], _dense(n.dNF[below]), acc=False)
        G = _dense(n.G["B"])
        c0 = n.P[n.levels].shape[3]
        self._block_bwd("B", G, c0, True, n.dNF["B"])
        dP_src = Slice(G.t, 0, G.ld, c0)
        for d in range(n.levels, 0, -1):
            # gradient of the pooled output -> dense, then through the pool
            # (gated by the transition's ReLU output) and the 1x1 conv, whose
            # input gradient is added to the skip's gradient already in place
            self.copy(f"P{d}.dy", dP_src, _dense(n.dP[d]))
            td = n.act[f"TD{d}"]
            self._add(f"TD{d}.dpool", "avg_pool2d_bwd_kernel", 2 * td.numel() * 9 // 4,
                      Lb.avg_pool2d_bwd,
                      (n.dP[d].data_ptr(), td.data_ptr(), *td.shape, n.dT[d].data_ptr()))
            Gu = n.G[f"U{d}"]
            G = Slice(Gu, nk, Gu.shape[3], n.inp[f"TD{d}"].ch)
            self.conv_bwd(f"TD{d}", n.inp[f"TD{d}"], n.dT[d], G, acc=True)
            c0 = n.L[f"D{d}.1"].x_shape[3]
            self._block_bwd(f"D{d}", G, c0, False)
            dP_src = Slice(G.t, G.off, G.ld, c0)
        c0 = n.L["C0"].y_shape[3]
        self.copy("C0.dy", dP_src, _dense(n.dC0), gate=n.out["C0"])
        self.conv_bwd("C0", _dense(n.x), n.dC0, _dense(n.dX), acc=False)
        assert self._dw_seen == n.dw_order(), "kernel gradients out of completion order"

    def set_loss_scale(self, s):
        self.net.loss_scale = float(s)
        self._head_args[3].value = s / self.net.act["F1x1"].numel()
        self._inv_scale.value = 1.0 / s

    def run(self, events=None, kernel_events=None):
        """Run the step once. events: {call index: (start, end)} HIP events
        recorded around those calls on the call's stream; kernel_events: the
        same for convolution calls, recorded by the library around the call's
        main kernel only."""
        streams, evs = self.streams, self.events
        for i, c in enumerate(self.calls):
            s = streams[c.sid]
            for d in c.deps:
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

    def join(self):
        """The main stream already waits for the other streams' last calls
        at the end of each run."""
