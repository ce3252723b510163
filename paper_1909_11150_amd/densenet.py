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

Dense concatenation: the convolution kernels read dense NHWC inputs, so a
block keeps one buffer per layer input, Z_l = concat(Z_{l-1}, Y_l), written
by two channel-slice copies. Backward, each block keeps a gradient buffer G
in the layout of its last concatenation: a layer's output gradient is its
slice of G, gated by its ReLU output; the layer's input gradient is added
into the slices it read. A skip connection's gradient (a slice of the up
block's G) is added to the down block's G, which the transition-down conv
writes first. fp16 storage throughout; every addition is one rounding.
"""
import ctypes

import torch

from . import (EPI_NONE, EPI_RELU, OP_BWD_DATA, OP_BWD_WEIGHT, OP_CONVT, OP_FWD,
               FgError, kernel_name, lib, workspace_bytes)
from .fcn import (Call, chain_workspace_bytes, convt_dw_desc, convt_dx_desc, fwd_desc,
                  kernel_gradient_workspace_bytes)

F16 = torch.float16


def _structure(layers):
    names = [L.name for L in layers]
    levels = sum(1 for n in names if n.startswith("TD"))
    per = sum(1 for n in names if n.startswith("B."))
    for req in ["C0", "F1x1"] + [f"TD{d}" for d in range(1, levels + 1)] + \
               [f"TU{d}" for d in range(1, levels + 1)]:
        if req not in names:
            raise ValueError(f"layer {req} missing from the dense network")
    return levels, per


class DenseNet:
    def __init__(self, layers, weights, x, loss_scale=2.0 ** 15, delta=10.0,
                 device="cuda", stream=None):
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
        self.act = {L.name: e(L.y_shape) for L in self.layers}   # post-ReLU outputs
        self.ws = torch.empty(max(chain_workspace_bytes(self.layers), 16),
                              dtype=torch.uint8, device=self.dev)
        # forward buffers: Z[(block, l)] = input of layer l + 1 of the block
        # (l = 0: the block input), pooled outputs, new-feature buffers
        self.Z, self.P, self.NF = {}, {}, {}
        self.G, self.dNF = {}, {}
        for d in range(1, self.levels + 1):
            self._block_bufs(f"D{d}")
            td = self.L[f"TD{d}"]
            n, h, w, c = td.y_shape
            self.P[d] = e((n, h // 2, w // 2, c))
        self._block_bufs("B")
        for d in range(1, self.levels + 1):
            self._block_bufs(f"U{d}")
        # gradient buffers (the input-gradient scratch dZin is one per
        # resolution: the main stream uses it in order)
        self.g_out = e(self.L["F1x1"].y_shape)
        self.dX = e(self.x.shape)
        # a layer's output gradient has a buffer of its own: its kernel
        # gradient may still read it on the side stream while the next
        # layer's is written
        self.dY, self.dZin, self.dT, self.dP, self.dU = {}, {}, {}, {}, {}
        for blk in self._blocks():
            n, h, w, _ = self.L[f"{blk}.1"].x_shape
            cmax = max(self.L[f"{blk}.{l}"].x_shape[3] for l in range(1, self.per + 1))
            for l in range(1, self.per + 1):
                self.dY[f"{blk}.{l}"] = e((n, h, w, self.k))
            old = self.dZin.get(h)
            if old is None or old.shape[3] < cmax:
                self.dZin[h] = e((n, h, w, cmax))
        for d in range(1, self.levels + 1):
            self.dT[d] = e(self.L[f"TD{d}"].y_shape)
            n, h, w, c = self.L[f"TD{d}"].y_shape
            self.dP[d] = e((n, h // 2, w // 2, c))
            self.dU[d] = e(self.L[f"TU{d}"].y_shape)
        self.dC0 = e(self.L["C0"].y_shape)
        self._L = lib()

    def _blocks(self):
        return [f"D{d}" for d in range(1, self.levels + 1)] + ["B"] + \
               [f"U{d}" for d in range(1, self.levels + 1)]

    def _block_bufs(self, blk):
        e = lambda s: torch.empty(s, dtype=F16, device=self.dev)
        n, h, w, c0 = self.L[f"{blk}.1"].x_shape
        if blk.startswith("U"):           # block input: concat(TU out, skip)
            self.Z[(blk, 0)] = e((n, h, w, c0))
        # the last concatenation is read only where it is a skip (down blocks)
        last = self.per if blk.startswith("D") else self.per - 1
        for l in range(1, last + 1):
            self.Z[(blk, l)] = e((n, h, w, c0 + l * self.k))
        self.G[blk] = e((n, h, w, c0 + self.per * self.k))
        if not blk.startswith("D"):
            self.NF[blk] = e((n, h, w, self.per * self.k))
            self.dNF[blk] = e((n, h, w, self.per * self.k))

    # ---- prepared calls ----------------------------------------------------------
    def program(self, target, streams=2):
        """streams = 1: every call in order on one stream; 2: the kernel
        gradients on a second stream; 3: also the forward pass's
        concatenation copies that do not wait for the layer they follow on a
        third. Measured on the full network: 6.73, 6.51 and 6.70 ms per step
        (the copy stream slows the forward convolutions it runs beside by
        more than it saves), so 2 is the default."""
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
    With three, the copy of a dense layer's input into the prefix of its
    block's next concatenation, and of its output into the block's
    new-feature buffer, run on the third beside the layer's convolution
    (each after the calls that complete what it reads; the convolution that
    reads a concatenation waits for both of its copies). The main stream
    waits for the other streams' last calls at the end of the step, before
    the next forward pass overwrites what they read. Every kernel reads only
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
        if streams > 1:
            self._ws_side = torch.empty(
                max(16, kernel_gradient_workspace_bytes(net.layers)), dtype=torch.uint8,
                device=net.dev)
        self._build(target)
        if streams == 1:
            self.calls = [c._replace(sid=0, deps=()) for c in self.calls]
        # a dependency on a call of the same stream is its stream order
        self.calls = [c._replace(deps=tuple(d for d in c.deps if self.calls[d].sid != c.sid))
                      for c in self.calls]
        self.calls = [c._replace(args=c.args + (self._sp[c.sid],)) for c in self.calls]
        self.final = tuple(max(j for j, c in enumerate(self.calls) if c.sid == sid)
                           for sid in range(1, len(self.streams)))
        self.step_final = self.final
        needed = {d for c in self.calls for d in c.deps} | set(self.final)
        self.events = {j: torch.cuda.Event() for j in sorted(needed)}

    # -- checks: every buffer a call touches holds what the call addresses --
    @staticmethod
    def _span_ok(t, off, ld, npix, nch):
        need = off + (npix - 1) * ld + nch
        if t.dtype != F16 or not t.is_contiguous() or t.numel() < need:
            raise ValueError(f"buffer of {t.numel()} fp16 elements, call reaches {need}")

    @staticmethod
    def _shape_ok(t, shape):
        if tuple(t.shape) != tuple(shape) or not t.is_contiguous():
            raise ValueError(f"tensor {tuple(t.shape)} where {tuple(shape)} is needed")

    def _desc(self, d):
        self._keep.append(d)
        return ctypes.byref(d)

    def _add(self, label, kernel, work, fn, args, single=True, sid=0, deps=()):
        """Append a call; the stream argument is added once all are built."""
        self.calls.append(Call(label, kernel, work, fn, args, single, sid, deps))

    # -- ops --
    def conv_fwd(self, name, x, y, relu, deps=()):
        L = self.net.L[name]
        n = self.net
        self._shape_ok(x, L.x_shape)
        self._shape_ok(y, L.y_shape)
        d = fwd_desc(L)
        epi = EPI_RELU if relu else EPI_NONE
        if L.kind == "conv":
            self._add(f"{name}.fwd", kernel_name(d, OP_FWD), L.flops, self._L.conv2d_fwd,
                      (self._desc(d), x.data_ptr(), n.w[name].data_ptr(), y.data_ptr(), epi,
                       None, n.ws.data_ptr(), n.ws.numel()),
                      workspace_bytes(d, OP_FWD) == 0, deps=deps)
        else:
            self._add(f"{name}.fwd", kernel_name(d, OP_CONVT), L.flops,
                      self._L.conv_transpose2d_fwd,
                      (self._desc(d), x.data_ptr(), n.w[name].data_ptr(), y.data_ptr(), epi,
                       None, n.ws.data_ptr(), n.ws.numel()),
                      workspace_bytes(d, OP_CONVT) == 0, deps=deps)

    def conv_bwd(self, name, x, dy, dx):
        """Kernel gradient into dw[name] (second stream, after the call that
        wrote dy, which is the last one appended); input gradient into dx
        (no gate)."""
        L = self.net.L[name]
        n = self.net
        self._shape_ok(x, L.x_shape)
        self._shape_ok(dy, L.y_shape)
        self._shape_ok(dx, L.x_shape)
        wsp, wsb = n.ws.data_ptr(), n.ws.numel()
        side = len(self.streams) > 1
        dws, dwb = (self._ws_side.data_ptr(), self._ws_side.numel()) if side else (wsp, wsb)
        dwk = dict(sid=self._dw_sid, deps=(len(self.calls) - 1,))
        if L.kind == "conv":
            d = fwd_desc(L)
            self._add(f"{name}.dW", kernel_name(d, OP_BWD_WEIGHT), L.flops,
                      self._L.conv2d_bwd_weight,
                      (self._desc(d), x.data_ptr(), dy.data_ptr(), n.dw[name].data_ptr(),
                       dws, dwb), workspace_bytes(d, OP_BWD_WEIGHT) == 0, **dwk)
            self._add(f"{name}.dx", kernel_name(d, OP_BWD_DATA), L.flops,
                      self._L.conv2d_bwd_data,
                      (self._desc(d), dy.data_ptr(), n.w[name].data_ptr(), dx.data_ptr(),
                       EPI_NONE, None, wsp, wsb), workspace_bytes(d, OP_BWD_DATA) == 0)
        else:
            d = convt_dw_desc(L)
            self._add(f"{name}.dW", kernel_name(d, OP_BWD_WEIGHT), L.flops,
                      self._L.conv2d_bwd_weight,
                      (self._desc(d), dy.data_ptr(), x.data_ptr(), n.dw[name].data_ptr(),
                       dws, dwb), workspace_bytes(d, OP_BWD_WEIGHT) == 0, **dwk)
            d = convt_dx_desc(L)
            self._add(f"{name}.dx", kernel_name(d, OP_FWD), L.flops, self._L.conv2d_fwd,
                      (self._desc(d), dy.data_ptr(), n.w[name].data_ptr(), dx.data_ptr(),
                       EPI_NONE, None, wsp, wsb), workspace_bytes(d, OP_FWD) == 0)

    def copy(self, label, src, soff, sld, dst, doff, dld, nch, gate=None, gld=0,
             acc=False, sid=0, deps=()):
        """nch channels per pixel; the pixel count is dst's over its stride."""
        npix = dst.numel() // dld
        self._span_ok(src, soff, sld, npix, nch)
        self._span_ok(dst, doff, dld, npix, nch)
        if gate is not None:
            self._span_ok(gate, 0, gld, npix, nch)
        rd = 2 * nch * npix * (2 if acc else 1) + (2 * nch * npix if gate is not None else 0)
        self._add(label, f"channel_slice_copy_kernel<{'true' if acc else 'false'}>",
                  rd + 2 * nch * npix, self._L.channel_slice_copy,
                  (src.data_ptr() + 2 * soff, sld,
                   None if gate is None else gate.data_ptr(), gld,
                   dst.data_ptr() + 2 * doff, dld, npix, nch, int(acc)),
                  sid=sid, deps=deps)
        return len(self.calls) - 1

    # -- the step --
    def _block_fwd(self, blk, z0, ready):
        """Dense layers of a block whose input z0 is complete once the calls
        in `ready` are. Returns the last concatenation (down blocks) and the
        calls that complete it; for other blocks, the calls that complete
        the new-feature buffer."""
        n = self.net
        z = z0
        nf_ready = []
        for l in range(1, n.per + 1):
            name = f"{blk}.{l}"
            self.conv_fwd(name, z, n.act[name], True, deps=ready)
            conv = len(self.calls) - 1
            if not blk.startswith("D"):     # new features: the block's outputs
                nf_ready.append(self.copy(f"{name}.new", n.act[name], 0, n.k, n.NF[blk],
                                          (l - 1) * n.k, n.per * n.k, n.k,
                                          sid=self._cp_sid, deps=(conv,)))
            if (blk, l) not in n.Z:
                continue
            out = n.Z[(blk, l)]
            cz, co = z.shape[3], out.shape[3]
            cat0 = self.copy(f"{name}.cat0", z, 0, cz, out, 0, co, cz,
                             sid=self._cp_sid, deps=ready)
            cat1 = self.copy(f"{name}.cat1", n.act[name], 0, n.k, out, cz, co, n.k)
            z, ready = out, (cat0, cat1)
        return (z, ready) if blk.startswith("D") else tuple(nf_ready)

    def _block_bwd(self, blk, fresh):
        """G[blk] holds the gradient of the block's last concatenation (for a
        fresh block only its new-feature channels); leaves the gradient of
        the block input in G[blk][..., :c0]."""
        n = self.net
        G = n.G[blk]
        cl = G.shape[3]
        c0 = n.L[f"{blk}.1"].x_shape[3]
        for l in range(n.per, 0, -1):
            name = f"{blk}.{l}"
            lo = c0 + (l - 1) * n.k
            h = n.L[name].x_shape[1]
            dY = n.dY[name]
            zin = n.Z[(blk, l - 1)] if l > 1 or blk.startswith("U") else self._block_input[blk]
            self.copy(f"{name}.dy", G, lo, cl, dY, 0, n.k, n.k, gate=n.act[name], gld=n.k)
            dZ = n.dZin[h]
            dZv = dZ.view(-1)[:zin.numel()].view(zin.shape)
            self.conv_bwd(name, zin, dY, dZv)
            if fresh and l == n.per:  # the block input's slice of G is still empty
                self.copy(f"{name}.dz0", dZv, 0, lo, G, 0, cl, c0)
                if lo > c0:
                    self.copy(f"{name}.dzacc", dZv, c0, lo, G, c0, cl, lo - c0, acc=True)
            else:
                self.copy(f"{name}.dzacc", dZv, 0, lo, G, 0, cl, lo, acc=True)

    def _build(self, target):
        n = self.net
        Lb = self._L
        self._block_input = {}
        # forward
        self.conv_fwd("C0", n.x, n.act["C0"], True)
        bin_, ready = n.act["C0"], (len(self.calls) - 1,)
        skips, skip_ready = {}, {}
        for d in range(1, n.levels + 1):
            self._block_input[f"D{d}"] = bin_
            z, zr = self._block_fwd(f"D{d}", bin_, ready)
            skips[d], skip_ready[d] = z, zr
            self.conv_fwd(f"TD{d}", z, n.act[f"TD{d}"], True, deps=zr)
            td = n.act[f"TD{d}"]
            self._add(f"TD{d}.pool", "avg_pool2d_fwd_kernel", 2 * td.numel() * 5 // 4,
                      Lb.avg_pool2d_fwd,
                      (td.data_ptr(), *td.shape, n.P[d].data_ptr()))
            bin_, ready = n.P[d], (len(self.calls) - 1,)
        self._block_input["B"] = bin_
        nf_ready = self._block_fwd("B", bin_, ready)
        nf = n.NF["B"]
        self._tu_in = {}
        for d in range(n.levels, 0, -1):
            tu = f"TU{d}"
            self._tu_in[d] = nf
            self.conv_fwd(tu, nf, n.act[tu], True, deps=nf_ready)
            z0 = n.Z[(f"U{d}", 0)]
            nk, c0 = n.act[tu].shape[3], z0.shape[3]
            cat1 = self.copy(f"{tu}.cat1", skips[d], 0, skips[d].shape[3], z0, nk, c0,
                             c0 - nk, sid=self._cp_sid, deps=skip_ready[d])
            cat0 = self.copy(f"{tu}.cat0", n.act[tu], 0, nk, z0, 0, c0, nk)
            nf_ready = self._block_fwd(f"U{d}", z0, (cat0, cat1))
            nf = n.NF[f"U{d}"]
        y = n.act["F1x1"]
        self.conv_fwd("F1x1", nf, y, False, deps=nf_ready)
        # head: loss-scaled mean Huber loss
        self._head_args = [y.data_ptr(), target.data_ptr(), y.numel(),
                           ctypes.c_double(n.loss_scale / y.numel()),
                           ctypes.c_double(n.delta), n.g_out.data_ptr()]
        self._add("head_grad", "huber_head_grad_kernel", 10 * y.numel(),
                  Lb.huber_head_grad, tuple(self._head_args))
        # backward: head, up blocks (level 1 first), bottleneck, down path
        self.conv_bwd("F1x1", nf, n.g_out, n.dNF["U1"])
        up_skip = {}
        for d in range(1, n.levels + 1):
            blk = f"U{d}"
            G = n.G[blk]
            cl, c0 = G.shape[3], n.L[f"{blk}.1"].x_shape[3]
            self.copy(f"{blk}.dnew", n.dNF[blk], 0, n.per * n.k, G, c0, cl, n.per * n.k)
            self._block_bwd(blk, fresh=True)
            tu = f"TU{d}"
            nk = n.per * n.k
            self.copy(f"{tu}.dy", G, 0, cl, n.dU[d], 0, nk, nk, gate=n.act[tu], gld=nk)
            below = "B" if d == n.levels else f"U{d + 1}"
            self.conv_bwd(tu, self._tu_in[d], n.dU[d], n.dNF[below])
            up_skip[d] = (G, nk, cl)
        G = n.G["B"]
        cl, c0 = G.shape[3], n.L["B.1"].x_shape[3]
        self.copy("B.dnew", n.dNF["B"], 0, n.per * n.k, G, c0, cl, n.per * n.k)
        self._block_bwd("B", fresh=True)
        dP_src, dP_off, dP_ld = G, 0, cl
        for d in range(n.levels, 0, -1):
            # gradient of the pooled output -> dense, then through the pool
            # (gated by the transition's ReLU output) and the 1x1 conv
            c = n.P[d].shape[3]
            self.copy(f"P{d}.dy", dP_src, dP_off, dP_ld, n.dP[d], 0, c, c)
            td = n.act[f"TD{d}"]
            self._add(f"TD{d}.dpool", "avg_pool2d_bwd_kernel", 2 * td.numel() * 9 // 4,
                      Lb.avg_pool2d_bwd,
                      (n.dP[d].data_ptr(), td.data_ptr(), *td.shape, n.dT[d].data_ptr()))
            blk = f"D{d}"
            G = n.G[blk]
            self.conv_bwd(f"TD{d}", skips[d], n.dT[d], G)
            Gu, off, ldu = up_skip[d]
            self.copy(f"{blk}.dskip", Gu, off, ldu, G, 0, G.shape[3], G.shape[3], acc=True)
            self._block_bwd(blk, fresh=False)
            dP_src, dP_off, dP_ld = G, 0, G.shape[3]
        c0 = n.act["C0"].shape[3]
        self.copy("C0.dy", dP_src, 0, dP_ld, n.dC0, 0, c0, c0, gate=n.act["C0"], gld=c0)
        self.conv_bwd("C0", n.x, n.dC0, n.dX)

    def set_loss_scale(self, s):
        self.net.loss_scale = float(s)
        self._head_args[3].value = s / self.net.act["F1x1"].numel()

    def run(self, events=None):
        """Run the step once. events: {call index: (start, end)} HIP events
        recorded around those calls on the call's stream."""
        streams, evs = self.streams, self.events
        for i, c in enumerate(self.calls):
            s = streams[c.sid]
            for d in c.deps:
                s.wait_event(evs[d])
            ev = events.get(i) if events else None
            if ev:
                ev[0].record(s)
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
        """The main stream already waits for the other stream's last call
        at the end of each run."""
