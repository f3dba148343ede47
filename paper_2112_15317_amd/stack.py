"""Host-side step drivers: buffer plan and call sequence of one worker step.

A worker of the paper's hybrid scheme runs the convolutional layers on its
local batch (data parallel) and its FC column shards on the batch gathered
from all replicas (model parallel); backward retraces the same path (sec.
3.1 and sec. 4).  These classes own the device buffers of that step and
enqueue the libsb calls in order (the conv weight gradients on a second
stream, see ``ConvStack``).  They do no arithmetic: every value is produced
by a libsb kernel.  torch only allocates device memory and orders streams.

``ConvStack``   13-layer VGG conv stack fwd + bwd (ReLU, fused ReLU + pool)
``FCShard``     one FC column shard fwd + bwd
``HybridStep``  conv stack, then FC0 -> ReLU -> FC1 shards on the gathered
                batch, then backward through both
``GroupTrainStep``  a training step of an MP group: conv stack, K modulo
                iterations of the FC shards with an update after each, conv
                backward and update
"""
from __future__ import annotations

import re

import numpy as np
import torch

from . import sb
from .configs import conv_layers


def _dev_dtype(dtype: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def _code(dtype: str):
    return {"f32": sb.SB_F32, "bf16": sb.SB_BF16}[dtype]


def _plain(key, fn, *args):
    fn(*args)


def capture_graph(step_fn, steps=1):
    """Record `steps` calls of step_fn into a HIP graph (through torch's
    graph capture: libsb enqueues on the current stream, which is the
    capturing one).  Launch-bound sequences of small kernels then replay with
    no per-launch host cost.  step_fn must have run eagerly once before, so
    that one-time kernel attribute setup happens outside the capture."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(steps):
            step_fn()
    return g


class ConvStack:
    """Buffers and calls of a 3x3 conv stack whose last layer is pooled.

    Buffer names (per layer l, 0-based):
      A[l]   input of layer l (A[0] = images, A[L] = stack output)
      Z[l]   pre-pool conv output of a pooled layer
      idx[l] pool window codes of a pooled layer
      gA[l]  gradient arriving at A[l] (gA[L] = upstream gradient); when
             layer l-1 has no pool, gA[l] already carries its ReLU mask,
             i.e. it is the gradient of that layer's conv output
      dZ[l]  gradient at the conv output of a pooled layer (pool backward)
      dW[l], db[l]  fp32 parameter gradients

    overlap: in backward the weight gradient of each layer runs on a second
    stream, forked after its output gradient is ready and joined at the end,
    so it overlaps the data-gradient chain (the two only share inputs, and
    each has its own split-reduction workspace).  Off by default: the large
    kernels are planned as one full round of blocks over the CUs (two per
    CU), so a kernel running beside one pushes some of its blocks into a
    second round; on the fp32 CIFAR step the overlapped backward is about 5 %
    slower than one stream, on the bf16 ImageNet-shaped step about 1 %
    faster.
    """

    def __init__(self, schedule, n, in_ch, hw, dtype="f32", device="cuda",
                 out_buffer=None, out_grad_buffer=None, packed=True, overlap=False,
                 layout="nchw", fuse_pool=True, batch_wgrad=True):
        """layout: "nchw", or "c8" for channel-blocked activations
        (SB_NCHW8C, bf16 only): every activation buffer is then
        [n][c/8][h][w][8], and the first layer's input channels are padded
        with zeros to a whole block of 8 (zero filters for the padding, so
        every result is the unpadded network's).

        fuse_pool: a pooled layer whose forward can pool in the kernel
        (sb_conv3x3_fwd_pool takes its descriptor: channel-blocked bf16 or
        NCHW fp32, an unsplit plan) runs its forward, ReLU and pooling as one
        call and has no Z buffer (``self.fused`` lists those layers).

        batch_wgrad: consecutive layers whose weight gradients run on the same
        fp32 kernel (``group_wgrads``) have them issued together, by one
        sb_conv3x3_bwd_weight_many call at the group's last layer (nothing in
        the step reads dW before the update), as one launch instead of one
        per layer (``self.wg_groups``)."""
        self.layers = conv_layers(schedule, in_ch, hw)
        if not self.layers[-1].pool_after:
            raise ValueError("the stack must end with a pooled layer")
        if layout not in ("nchw", "c8") or (layout == "c8" and dtype != "bf16"):
            raise ValueError("layout 'c8' is for bf16 stacks")
        if layout == "c8" and min(l.w for l in self.layers) < 8:
            raise ValueError("layout 'c8' needs images at least 8 wide at every layer")
        self.n, self.dtype = n, dtype
        self.code = _code(dtype)
        self.c8 = layout == "c8"
        self.layout = sb.SB_NCHW8C if self.c8 else sb.SB_NCHW
        tdt = _dev_dtype(dtype)
        dev = torch.device(device)
        self.device = dev
        L = self.layers
        # Input channels of each layer as stored (the first padded for c8).
        self.cin = [(-(-l.c // 8) * 8 if self.c8 else l.c) for l in L]
        shp = self.shape_of
        self.A = [torch.empty(shp(n, self.cin[0], hw, hw), dtype=tdt, device=dev)]
        self.Z, self.idx, self.dZ = {}, {}, {}
        for l in L:
            if l.pool_after:
                self.Z[l.index] = torch.empty(shp(n, l.k, l.h, l.w), dtype=tdt, device=dev)
                self.idx[l.index] = torch.empty(shp(n, l.k, l.h // 2, l.w // 2),
                                                dtype=torch.uint8, device=dev)
                self.dZ[l.index] = torch.empty(shp(n, l.k, l.h, l.w), dtype=tdt, device=dev)
                shape = shp(n, l.k, l.h // 2, l.w // 2)
            else:
                shape = shp(n, l.k, l.h, l.w)
            last = l.index == len(L) - 1
            if last and out_buffer is not None:
                self.A.append(out_buffer.view(shape))
            else:
                self.A.append(torch.empty(shape, dtype=tdt, device=dev))
        self.gA = [torch.empty_like(a) for a in self.A[:-1]]
        self.gA.append(out_grad_buffer.view(self.A[-1].shape) if out_grad_buffer is not None
                       else torch.empty_like(self.A[-1]))
        C = self.cin
        lay = self.layout
        # Pooled layers that pool inside the forward (their Z is never stored).
        self.fused = (self.fused_layers(schedule, n, in_ch, hw, dtype, layout, packed)
                      if fuse_pool else set())
        for i in self.fused:
            del self.Z[i]
        self.W = [torch.zeros((l.k, C[l.index], 3, 3), dtype=tdt, device=dev) for l in L]
        self.b = [torch.zeros((l.k,), dtype=torch.float32, device=dev) for l in L]
        self.dW = [torch.empty((l.k, C[l.index], 3, 3), dtype=torch.float32, device=dev)
                   for l in L]
        self.db = [torch.empty((l.k,), dtype=torch.float32, device=dev) for l in L]
        self.desc = [sb.conv_desc(n, C[l.index], l.h, l.w, l.k, self.code, relu=not l.pool_after,
                                  layout=lay) for l in L]
        self.desc_b = [sb.conv_desc(n, C[l.index], l.h, l.w, l.k, self.code, layout=lay)
                       for l in L]
        # packed: every layer's filters are packed for the forward and the
        # data-gradient pass in one launch at the start of the step
        # (sb_conv3x3_pack_filters_many), and the passes take them with
        # SB_PACKED_FILTERS, instead of each pass packing its own ahead of it
        # (26 small launches on VGG-16, each mostly ramp-up and drain).
        self.packed = packed
        self.pdesc = self.desc
        self.pdesc_b = self.desc_b
        if packed:
            self.pdesc = [sb.conv_desc(n, C[l.index], l.h, l.w, l.k, self.code,
                                       relu=not l.pool_after, packed=True, layout=lay)
                          for l in L]
            self.pdesc_b = [sb.conv_desc(n, C[l.index], l.h, l.w, l.k, self.code, packed=True,
                                         layout=lay) for l in L]

            def buf(i, pass_):
                nb = sb.sb_conv3x3_packed_bytes(self.desc_b[i], pass_)
                return torch.empty((max(nb, 256),), dtype=torch.uint8, device=dev)
            self.Wf = [buf(l.index, sb.SB_PASS_FWD) for l in L]
            self.Wb = [buf(l.index, sb.SB_PASS_BWD_DATA) for l in L]
            self.packs = sb.PackList(
                [(self.desc_b[i], sb.SB_PASS_FWD, self.W[i], self.Wf[i]) for i in range(len(L))] +
                [(self.desc_b[i], sb.SB_PASS_BWD_DATA, self.W[i], self.Wb[i])
                 for i in range(len(L))])
        need = 0
        for l in L:
            need = max(need,
                       sb.sb_conv3x3_workspace_bytes(self.pdesc[l.index], sb.SB_PASS_FWD),
                       sb.sb_conv3x3_workspace_bytes(self.pdesc_b[l.index], sb.SB_PASS_BWD_DATA),
                       sb.sb_conv3x3_workspace_bytes(self.desc_b[l.index], sb.SB_PASS_BWD_WEIGHT))
        # Weight gradients batched into one call per group (layers in
        # backward order); each group's call needs the sum of its layers'
        # workspace regions.
        self.wg_groups = self.group_wgrads([self.desc_b[l.index] for l in L]) if batch_wgrad \
            else []
        self.wg_group_of = {}
        self.wg_lists = {}
        for grp in self.wg_groups:
            for i in grp:
                self.wg_group_of[i] = grp
            self.wg_lists[grp[0]] = sb.WgradList(
                [self.desc_b[i] for i in grp], [self.A[i] for i in grp],
                [self.grad_at_conv_output(i) for i in grp], [self.dW[i] for i in grp],
                [self.db[i] for i in grp])
            need = max(need, self.wg_lists[grp[0]].workspace_bytes())
        # Split-reduction scratch; needs no initialisation.
        self.ws = torch.empty((max(need, 256) + 255) // 256 * 256, dtype=torch.uint8, device=dev)
        self.overlap = overlap and dev.type == "cuda"
        self.ws_w = self.ws
        if self.overlap:
            need_w = max([sb.sb_conv3x3_workspace_bytes(self.desc_b[l.index], sb.SB_PASS_BWD_WEIGHT)
                          for l in L] + [w.workspace_bytes() for w in self.wg_lists.values()])
            self.ws_w = torch.empty((max(need_w, 256) + 255) // 256 * 256, dtype=torch.uint8,
                                    device=dev)
            self.side = torch.cuda.Stream(device=dev)     # default priority
        self.call = _plain      # hook: every libsb call of the step goes through it

    @staticmethod
    def fused_layers(schedule, n, in_ch, hw, dtype="f32", layout="nchw", packed=True):
        """Indices of the pooled layers whose forward pools in the kernel
        (sb_conv3x3_fwd_pool takes their descriptor): host-side queries only."""
        c8 = layout == "c8"
        out = set()
        for l in conv_layers(schedule, in_ch, hw):
            c = -(-l.c // 8) * 8 if c8 else l.c
            d = sb.conv_desc(n, c, l.h, l.w, l.k, _code(dtype), packed=packed,
                             layout=sb.SB_NCHW8C if c8 else sb.SB_NCHW)
            if l.pool_after and \
                    sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD_POOL) != sb.SIZE_MAX:
                out.add(l.index)
        return out

    @staticmethod
    def group_wgrads(descs, most=4):
        """Groups (of two or more, at most `most`) of consecutive layers, in
        backward order, whose weight gradients run on the same fp32 wide-tile
        kernel, which sb_conv3x3_bwd_weight_many then issues as one launch:
        host-side queries only."""
        def name(d):
            s = sb.sb_conv3x3_plan_string(d, sb.SB_PASS_BWD_WEIGHT).split(" grid=")[0]
            return s if re.fullmatch(r"sb::conv3x3_wgrad_f32<sb::WgTile<\d+, \d+, \d+, 0>, float>",
                                     s) else None
        groups, run = [], []
        for i in reversed(range(len(descs))):
            nm = name(descs[i])
            if run and (nm is None or nm != name(descs[run[0]]) or len(run) == most):
                if len(run) > 1:
                    groups.append(run)
                run = []
            if nm is not None:
                run.append(i)
        if len(run) > 1:
            groups.append(run)
        return groups

    # -- layouts -----------------------------------------------------------------
    def shape_of(self, n, c, h, w):
        """Buffer shape of an activation of c channels in this stack's layout."""
        return (n, c // 8, h, w, 8) if self.c8 else (n, c, h, w)

    def to_layout(self, a, c=None):
        """A host NCHW array or tensor as a CPU tensor in this stack's layout
        (channels zero-padded to c)."""
        t = a if isinstance(a, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(a))
        if not self.c8:
            return t
        n, ch, h, w = t.shape
        c = c or ch
        if c != ch:
            t = torch.cat([t, torch.zeros((n, c - ch, h, w), dtype=t.dtype)], dim=1)
        return t.reshape(n, c // 8, 8, h, w).permute(0, 1, 3, 4, 2).contiguous()

    def nchw(self, t):
        """A device buffer of this stack as an NCHW tensor (a copy for c8)."""
        if not self.c8:
            return t
        n, cb, h, w, e = t.shape
        return t.permute(0, 1, 4, 2, 3).reshape(n, cb * e, h, w)

    # -- data placement (host -> device copies of seeded inputs) --------------
    def load_inputs(self, x, weights, biases=None, dy_top=None):
        def put(dst, t):
            dst.copy_(t.to(dst.dtype) if t.dtype != dst.dtype else t)
        put(self.A[0], self.to_layout(x, self.cin[0]))
        for l, w in enumerate(weights):
            t = w if isinstance(w, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(w))
            self.W[l].zero_()
            self.W[l][:, :t.shape[1]].copy_(t.to(self.W[l].dtype))
        if biases is not None:
            for l, b in enumerate(biases):
                t = b if isinstance(b, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(b))
                put(self.b[l], t)
        if dy_top is not None:
            put(self.gA[-1], self.to_layout(dy_top))

    # -- the step ---------------------------------------------------------------
    def forward(self, stream=None):
        c = self.call
        if self.packed:
            c(("pack", 0), sb.sb_conv3x3_pack_filters_many, self.packs, stream)
        for l in self.layers:
            i = l.index
            w = self.Wf[i] if self.packed else self.W[i]
            if i in self.fused:
                c(("fwd_pool", i), sb.sb_conv3x3_fwd_pool, self.pdesc_b[i], self.A[i], w,
                  self.b[i], self.A[i + 1], self.idx[i], self.ws, stream)
            elif l.pool_after:
                c(("fwd", i), sb.sb_conv3x3_fwd, self.pdesc[i], self.A[i], w, self.b[i],
                  self.Z[i], self.ws, stream)
                c(("pool_fwd", i), sb.sb_relu_maxpool_fwd, self.n, l.k, l.h, l.w, self.code,
                  self.layout, self.Z[i], self.A[i + 1], self.idx[i], stream)
            else:
                c(("fwd", i), sb.sb_conv3x3_fwd, self.pdesc[i], self.A[i], w, self.b[i],
                  self.A[i + 1], self.ws, stream)

    def backward(self, stream=None, want_dx=True):
        c = self.call
        L = self.layers
        # Two streams only for the real calls (a recorded call list, from
        # step_calls, stays stream-agnostic) and for a torch stream or the
        # current one (a raw stream handle cannot record events here).
        fork = (self.overlap and c is _plain and
                (stream is None or isinstance(stream, torch.cuda.Stream)))
        if fork:
            main = stream if stream is not None else torch.cuda.current_stream(self.device)
        for l in reversed(L):
            i = l.index
            if l.pool_after:
                c(("pool_bwd", i), sb.sb_relu_maxpool_bwd, self.n, l.k, l.h, l.w, self.code,
                  self.layout, self.gA[i + 1], self.idx[i], self.dZ[i], stream)
                g = self.dZ[i]
            else:
                g = self.gA[i + 1]
            ws_stream = stream
            grp = self.wg_group_of.get(i)
            if grp is None or i == grp[-1]:
                if fork:
                    ready = torch.cuda.Event()
                    ready.record(main)
                    self.side.wait_event(ready)
                    ws_stream = self.side
                if grp is None:
                    c(("wgrad", i), sb.sb_conv3x3_bwd_weight, self.desc_b[i], self.A[i], g,
                      self.dW[i], self.db[i], self.ws_w, ws_stream)
                else:
                    # The group's last layer: every member's output gradient
                    # is ready now.
                    c(("wgrad_many", grp[0]), sb.sb_conv3x3_bwd_weight_many,
                      self.wg_lists[grp[0]], self.ws_w, ws_stream)
            w = self.Wb[i] if self.packed else self.W[i]
            if i > 0:
                mask = None if L[i - 1].pool_after else self.A[i]
                c(("dgrad", i), sb.sb_conv3x3_bwd_data, self.pdesc_b[i], g, w, mask,
                  self.gA[i], self.ws, stream)
            elif want_dx:
                c(("dgrad", i), sb.sb_conv3x3_bwd_data, self.pdesc_b[i], g, w, None,
                  self.gA[0], self.ws, stream)
        if fork:
            done = torch.cuda.Event()
            done.record(self.side)
            main.wait_event(done)

    def grad_at_conv_output(self, i):
        """Gradient at conv output i (after its ReLU / pool backward)."""
        return self.dZ[i] if self.layers[i].pool_after else self.gA[i + 1]

    def step(self, stream=None):
        self.forward(stream)
        self.backward(stream)

    def step_calls(self):
        """The ordered (key, libsb function, args) calls of one step."""
        rec = []
        saved = self.call
        self.call = lambda key, fn, *args: rec.append((key, fn, args))
        try:
            self.step()
        finally:
            self.call = saved
        return rec


class FCShard:
    """One FC column shard: X [m, k_in] (row stride ldx), W [k_in, ns]."""

    def __init__(self, m, k_in, ns, relu=False, ldx=None, ldy=None, device="cuda"):
        self.m, self.k_in, self.ns, self.relu = m, k_in, ns, relu
        self.ldx, self.ldy = ldx or k_in, ldy or ns
        dev = torch.device(device)
        self.desc_f = sb.fc_desc(m, k_in, ns, sb.SB_F32, self.ldx, self.ldy, relu=relu)
        self.desc_b = sb.fc_desc(m, k_in, ns, sb.SB_F32, self.ldx, self.ldy)
        self.W = torch.empty((k_in, ns), dtype=torch.float32, device=dev)
        self.b = torch.zeros((ns,), dtype=torch.float32, device=dev)
        self.dW = torch.empty((k_in, ns), dtype=torch.float32, device=dev)
        self.db = torch.empty((ns,), dtype=torch.float32, device=dev)
        need = max(sb.sb_fc_workspace_bytes(self.desc_f, sb.SB_FC_FWD),
                   sb.sb_fc_workspace_bytes(self.desc_b, sb.SB_FC_BWD))
        # Split-reduction scratch; needs no initialisation.
        self.ws = torch.empty((max(need, 256) + 255) // 256 * 256, dtype=torch.uint8, device=dev)

    def fwd_call(self, x_ptr, y_ptr, stream=None):
        """(libsb function, args) of the forward."""
        return sb.sb_fc_shard_fwd, (self.desc_f, x_ptr, self.W, self.b, y_ptr, self.ws, stream)

    def bwd_call(self, x_ptr, dy_ptr, mask_ptr, dx_ptr, accumulate=False, stream=None):
        """(libsb function, args) of the backward."""
        return sb.sb_fc_shard_bwd, (self.desc_b, x_ptr, self.W, dy_ptr, mask_ptr, dx_ptr,
                                    self.dW, self.db, accumulate, self.ws, stream)

    def forward(self, x_ptr, y_ptr, stream=None):
        fn, args = self.fwd_call(x_ptr, y_ptr, stream)
        fn(*args)

    def backward(self, x_ptr, dy_ptr, mask_ptr, dx_ptr, accumulate=False, stream=None):
        fn, args = self.bwd_call(x_ptr, dy_ptr, mask_ptr, dx_ptr, accumulate, stream)
        fn(*args)


class HybridStep:
    """Conv stack on the local batch, then L FC shards on the gathered batch.

    X[0] [R*n, F]: rows [0, n) are this replica's flattened conv output (the
    stack writes them in place, NCHW order per image), rows [n, R*n) hold the
    other replicas' rows.  X[j] [R*n, in_j] for j >= 1: columns [0, ns_{j-1})
    are FC j-1's shard output (written in place, ReLU), the rest hold the
    other shards' columns.  The last shard's output Y has no ReLU.  Backward:
    FC j's partial input gradient restricted to this shard's columns of the
    layer below is that layer's output gradient (masked by its ReLU inside
    the call); FC0's partial input gradient restricted to this replica's rows
    is the conv stack's upstream gradient.  The cross-worker sums are
    collectives, not part of this step.
    """

    def __init__(self, schedule, n, in_ch, hw, replicas, fc_shapes, shards, device="cuda"):
        """The last shard's output Y takes a given gradient dY; nothing is
        updated (the training step with its K modulo iterations is
        ``GroupTrainStep``)."""
        dev = torch.device(device)
        self.n, self.R = n, replicas
        m = n * replicas
        self.m, self.L = m, len(fc_shapes)
        self.ins = [fi for fi, _ in fc_shapes]
        self.ns = [fo // shards for _, fo in fc_shapes]
        for j in range(1, self.L):
            assert self.ins[j] == fc_shapes[j - 1][1]
        f32 = dict(dtype=torch.float32, device=dev)
        self.X = [torch.empty((m, fi), **f32) for fi in self.ins]
        self.dXp = [torch.empty((m, fi), **f32) for fi in self.ins]
        self.Y = torch.empty((m, self.ns[-1]), **f32)
        self.dY = torch.empty((m, self.ns[-1]), **f32)
        self.conv = ConvStack(schedule, n, in_ch, hw, "f32", device,
                              out_buffer=self.X[0][:n], out_grad_buffer=self.dXp[0][:n])
        top = self.conv.A[-1]
        assert int(np.prod(top.shape[1:])) == self.ins[0]
        last = self.L - 1
        self.fc = [FCShard(m, self.ins[j], self.ns[j], relu=j < last, ldx=self.ins[j],
                           ldy=self.ins[j + 1] if j < last else self.ns[-1], device=device)
                   for j in range(self.L)]
        self.call = _plain      # hook: every libsb call of the step goes through it

    # Two-layer names used by the tests of the four-replica worker step.
    X0 = property(lambda self: self.X[0])
    X1 = property(lambda self: self.X[1])
    dX0p = property(lambda self: self.dXp[0])
    dX1p = property(lambda self: self.dXp[1])
    fc0 = property(lambda self: self.fc[0])
    fc1 = property(lambda self: self.fc[1])

    def load_inputs(self, x, conv_w, conv_b, fc_w, fc_b, rows_remote, cols_remote, dy):
        """fc_w / fc_b: the shard weights and biases per layer; rows_remote:
        the other replicas' rows of X[0]; cols_remote[j-1]: the other shards'
        columns of X[j]; dy: the gradient of the last shard's output."""
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
        self.conv.load_inputs(x, conv_w, conv_b)
        for f, w, b in zip(self.fc, fc_w, fc_b):
            f.W.copy_(t(w))
            f.b.copy_(t(b))
        self.X[0][self.n:].copy_(t(rows_remote))
        for j in range(1, self.L):
            self.X[j][:, self.ns[j - 1]:].copy_(t(cols_remote[j - 1]))
        self.dY.copy_(t(dy))

    def step(self, stream=None):
        def c(key, call):
            fn, args = call
            self.call(key, fn, *args)
        self.conv.forward(stream)
        L = self.L
        X = [x.data_ptr() for x in self.X]
        for j in range(L):
            out = X[j + 1] if j + 1 < L else self.Y.data_ptr()
            c(("fc_fwd", j), self.fc[j].fwd_call(X[j], out, stream))
        for j in reversed(range(L)):
            # Output gradient of layer j: the last layer's (given), or layer
            # j+1's partial input gradient on this shard's columns (row
            # stride in_{j+1}), masked by layer j's ReLU output X[j+1][:, :ns_j].
            dy = self.dY.data_ptr() if j == L - 1 else self.dXp[j + 1].data_ptr()
            mask = None if j == L - 1 else X[j + 1]
            c(("fc_bwd", j), self.fc[j].bwd_call(X[j], dy, mask, self.dXp[j].data_ptr(),
                                                 stream=stream))
        self.conv.backward(stream)

    def step_calls(self):
        """The ordered (key, libsb function, args) calls of one step."""
        rec = []
        saved = self.call, self.conv.call
        self.call = self.conv.call = lambda key, fn, *args: rec.append((key, fn, args))
        try:
            self.step()
        finally:
            self.call, self.conv.call = saved
        return rec


class GroupTrainStep:
    """One training step of an MP group of K workers on one device (sec. 3.1,
    Modulo Layer and Shard Layer), with the FC side of every worker of the
    group and the conv stack of worker 0.

    The model-parallel part runs the call sequence of ``plan``
    (``partition.fc_plan`` of the partitioned layer list): the modulo layer,
    then split dense layers each followed by a shard layer, then the loss.
    Worker 0 runs its conv stack forward once and writes the flattened
    output into slot 0 of ``local`` [K][B][F]; slots 1 .. K-1 hold the conv
    outputs of the group's other workers (their own data-parallel stacks,
    given as inputs).  Then K modulo iterations k = 0 .. K-1 each

      * gather B rows, B/K from every worker (``sb_modulo_fwd``, block k);
      * run, for every worker r, its column shard of each dense layer
        (``sb_fc_shard_fwd``, ReLU fused), and after each layer the shard
        layer that assembles the full input of the next one from the K
        partitions (``sb_shard_fwd``; before the loss: the full logits);
      * evaluate log-softmax + NLL of the full logits against the labels of
        the gathered rows, averaged over the B rows (``sb_log_softmax_nll``);
      * backpropagate: the last shards take their columns of the logits'
        gradient (every worker evaluates the same loss), each shard layer
        sums the group's partial input gradients over every worker's slice
        (``sb_shard_bwd``), and the modulo layer sums the first layer's
        partial input gradients back into the local rows of block k
        (``sb_modulo_bwd``);
      * take an SGD step on every FC shard with its gradient divided by K
        (``sb_sgd_update``), so iteration k + 1 runs on the updated weights.

    After the K iterations slot 0 of ``dlocal`` holds the gradient of worker
    0's conv output over its whole local batch: the conv stack runs backward
    and takes one SGD step at rate lr.

    Buffers (j: dense layer, r: worker): ``W[j]``/``b[j]`` [K][in_j][ns_j] /
    [K][ns_j] (worker r's shard, fp32), ``dW[j]``/``db[j]`` their gradients,
    ``X[j]`` [B][in_j] the full input of layer j (``X[0]`` the gathered
    batch, ``X[L]`` the full logits), ``P[j]`` [K][B][ns_j] the shard
    outputs, ``dF[j]`` [K][B][in_j] every worker's partial input gradient,
    ``dP[j]`` [K][B][ns_j] the shard layers' sums, ``labels`` [K][B] (int32,
    the labels of iteration k's gathered rows), ``loss`` [K][B].
    """

    def __init__(self, schedule, n, in_ch, hw, plan, lr=0.01, device="cuda"):
        dev = torch.device(device)
        if not plan or plan[0][0] != "modulo" or plan[-1][0] != "loss":
            raise ValueError("the plan must run from a modulo layer to the loss")
        lin = [e for e in plan[1:-1] if e[0] == "linear"]
        shards = [e for e in plan[1:-1] if e[0] == "shard"]
        body = [e[0] for e in plan[1:-1]]
        if body != ["linear", "shard"] * len(lin):
            raise ValueError("every dense layer must be split and followed by a shard layer")
        K = lin[0][3] // lin[0][2]
        for (_, i, ns, full, _), (_, part, whole) in zip(lin, shards):
            if ns * K != full or (part, whole) != (ns, full):
                raise ValueError("inconsistent shard widths in the plan")
        if n % K:
            raise ValueError("the local batch must divide into K blocks")
        self.K, self.B, self.L, self.lr = K, n, len(lin), lr
        self.ins = [e[1] for e in lin]
        self.ns = [e[2] for e in lin]
        self.full = [e[3] for e in lin]
        self.relu = [e[4] for e in lin]
        self.F = plan[0][1]
        self.classes = plan[-1][1]
        if self.ins[0] != self.F or self.full[-1] != self.classes:
            raise ValueError("the plan's widths do not chain")
        for j in range(1, self.L):
            if self.ins[j] != self.full[j - 1]:
                raise ValueError("the plan's widths do not chain")
        f32 = dict(dtype=torch.float32, device=dev)
        K, B, F = self.K, self.B, self.F
        self.local = torch.empty((K, B, F), **f32)
        self.dlocal = torch.empty((K, B, F), **f32)
        self.conv = ConvStack(schedule, n, in_ch, hw, "f32", device,
                              out_buffer=self.local[0], out_grad_buffer=self.dlocal[0])
        if int(np.prod(self.conv.A[-1].shape[1:])) != F:
            raise ValueError("the conv stack's output does not have the plan's width")
        L = self.L
        self.W = [torch.empty((K, self.ins[j], self.ns[j]), **f32) for j in range(L)]
        self.b = [torch.empty((K, self.ns[j]), **f32) for j in range(L)]
        self.dW = [torch.empty_like(w) for w in self.W]
        self.db = [torch.empty_like(b) for b in self.b]
        self.X = [torch.empty((B, self.ins[j]), **f32) for j in range(L)]
        self.X.append(torch.empty((B, self.classes), **f32))
        self.P = [torch.empty((K, B, self.ns[j]), **f32) for j in range(L)]
        self.dF = [torch.empty((K, B, self.ins[j]), **f32) for j in range(L)]
        self.dP = [torch.empty((K, B, self.ns[j]), **f32) for j in range(L)]
        self.dZl = torch.empty((B, self.classes), **f32)
        self.labels = torch.zeros((K, B), dtype=torch.int32, device=dev)
        self.loss = torch.empty((K, B), **f32)
        self.mdesc = sb.modulo_desc(K, K, B, F)
        self.sdesc = [sb.shard_desc(K, K, B, self.ns[j]) for j in range(L)]
        # Forward writes each shard's output densely ([B][ns_j]); the last
        # layer's backward reads its columns of the full logits' gradient.
        self.fdesc = [sb.fc_desc(B, self.ins[j], self.ns[j], relu=self.relu[j]) for j in range(L)]
        self.bdesc = [sb.fc_desc(B, self.ins[j], self.ns[j],
                                 ldy=self.classes if j == L - 1 else self.ns[j])
                      for j in range(L)]
        need = 0
        for j in range(L):
            need = max(need, sb.sb_fc_workspace_bytes(self.fdesc[j], sb.SB_FC_FWD),
                       sb.sb_fc_workspace_bytes(self.bdesc[j], sb.SB_FC_BWD))
        self.ws = torch.empty((max(need, 256) + 255) // 256 * 256, dtype=torch.uint8, device=dev)
        self.sgd_fc = sb.SgdList([(self.W[j], self.dW[j], 1.0 / K) for j in range(L)] +
                                 [(self.b[j], self.db[j], 1.0 / K) for j in range(L)])
        c = self.conv
        self.sgd_conv = sb.SgdList([(c.W[i], c.dW[i], 1.0) for i in range(len(c.layers))] +
                                   [(c.b[i], c.db[i], 1.0) for i in range(len(c.layers))])
        self.call = _plain      # hook: every libsb call of the step goes through it

    def load_inputs(self, x, conv_w, conv_b, fc_w, fc_b, local_remote, labels):
        """fc_w / fc_b: the full dense layers ([in][out], [out]); worker r's
        shard is columns r*ns .. (r+1)*ns - 1.  local_remote [K-1][B][F]:
        the other workers' conv outputs; labels [K][B]."""
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
        self.conv.load_inputs(x, conv_w, conv_b)
        K = self.K
        for j in range(self.L):
            w = np.asarray(fc_w[j], np.float32).reshape(self.ins[j], K, self.ns[j])
            self.W[j].copy_(t(w.transpose(1, 0, 2)))
            self.b[j].copy_(t(np.asarray(fc_b[j], np.float32).reshape(K, self.ns[j])))
        if K > 1:
            self.local[1:].copy_(t(local_remote))
        self.labels.copy_(torch.from_numpy(np.ascontiguousarray(labels, dtype=np.int32)))

    def full_weights(self, j):
        """Layer j's full weight [in][out] on the host (the shards side by side)."""
        w = self.W[j].detach().cpu().numpy()
        return np.ascontiguousarray(w.transpose(1, 0, 2).reshape(self.ins[j], -1))

    def full_bias(self, j):
        return self.b[j].detach().cpu().numpy().reshape(-1)

    # -- the step ---------------------------------------------------------------
    def iteration(self, k, stream=None):
        """Modulo iteration k: forward, loss, backward and FC update."""
        c = self.call
        K, L = self.K, self.L
        c(("mfwd", k), sb.sb_modulo_fwd, self.mdesc, 0, k, self.local, self.X[0], None, stream)
        for j in range(L):
            for r in range(K):
                c(("fc_fwd", j), sb.sb_fc_shard_fwd, self.fdesc[j], self.X[j], self.W[j][r],
                  self.b[j][r], self.P[j][r], self.ws, stream)
            c(("sfwd", j), sb.sb_shard_fwd, self.sdesc[j], 0, self.P[j], self.X[j + 1], None,
              stream)
        c(("loss", k), sb.sb_log_softmax_nll, self.B, self.classes, self.X[L], self.labels[k],
          1.0 / self.B, None, self.loss[k], self.dZl, None, stream)
        for j in reversed(range(L)):
            for r in range(K):
                if j == L - 1:
                    dy = self.dZl.data_ptr() + 4 * r * self.ns[j]     # its columns of dZl
                else:
                    dy = self.dP[j][r]
                mask = self.P[j][r] if self.relu[j] else None
                c(("fc_bwd", j), sb.sb_fc_shard_bwd, self.bdesc[j], self.X[j], self.W[j][r], dy,
                  mask, self.dF[j][r], self.dW[j][r], self.db[j][r], False, self.ws, stream)
            if j > 0:
                c(("sbwd", j), sb.sb_shard_bwd, self.sdesc[j - 1], 0, self.dF[j], self.dP[j - 1],
                  None, None, stream)
            else:
                c(("mbwd", k), sb.sb_modulo_bwd, self.mdesc, 0, k, self.dF[0], self.dlocal,
                  None, None, stream)
        c(("sgd_fc", k), sb.sb_sgd_update, self.sgd_fc, self.lr, stream)

    def finish(self, stream=None):
        """Conv backward from the gathered local-row gradients, conv update."""
        self.conv.backward(stream)
        self.call(("sgd_conv", 0), sb.sb_sgd_update, self.sgd_conv, self.lr, stream)

    def step(self, stream=None):
        self.conv.forward(stream)
        for k in range(self.K):
            self.iteration(k, stream)
        self.finish(stream)

    def step_calls(self):
        """The ordered (key, libsb function, args) calls of one step."""
        rec = []
        saved = self.call, self.conv.call
        self.call = self.conv.call = lambda key, fn, *args: rec.append((key, fn, args))
        try:
            self.step()
        finally:
            self.call, self.conv.call = saved
        return rec


class AveragedGroups:
    """G MP groups (each a GroupTrainStep on its own data) whose models are
    averaged every ``period`` steps: the data parallelism across MP groups
    (sec. 4: every worker exchanges its parameters up to the modulo layer
    every few batches, and each FC shard is averaged with the same shard of
    the other groups; sec. 2: the reduce is the mean of the replicas).

    One device holds every group: group g's tensors are its own
    GroupTrainStep's buffers, and the average of each parameter tensor (every
    conv layer's filters and bias, every FC layer's [K][in][ns] shards and
    [K][ns] biases, shard r of group g beside shard r of every other group)
    is one ``sb_model_average_replicas`` call over the G buffers.  ``step``
    runs every group's training step, then, after steps period, 2 period,
    ..., the averages.
    """

    def __init__(self, schedule, n, in_ch, hw, plan, groups, period, lr=0.01, device="cuda"):
        if groups < 1 or groups > sb.SB_MAX_REPLICAS:
            raise ValueError("1 .. %d groups" % sb.SB_MAX_REPLICAS)
        if period < 1:
            raise ValueError("the averaging period is a positive number of steps")
        self.groups = [GroupTrainStep(schedule, n, in_ch, hw, plan, lr, device)
                       for _ in range(groups)]
        self.period = period
        self.steps_done = 0

        def params(gs):
            c = gs.conv
            return list(c.W) + list(c.b) + list(gs.W) + list(gs.b)
        per_group = [params(gs) for gs in self.groups]
        self.sets = [list(ts) for ts in zip(*per_group)]     # one entry per parameter tensor
        self.call = _plain      # hook: every libsb call goes through it

    def load_inputs(self, group_inputs, conv_w, conv_b, fc_w, fc_b):
        """group_inputs[g] = (x, local_remote, labels) of group g; every group
        starts from the same model."""
        if len(group_inputs) != len(self.groups):
            raise ValueError("one input set per group")
        for gs, (x, remote, labels) in zip(self.groups, group_inputs):
            gs.load_inputs(x, conv_w, conv_b, fc_w, fc_b, remote, labels)

    def average(self, stream=None):
        for i, ts in enumerate(self.sets):
            self.call(("avg", i), sb.sb_model_average_replicas, ts, None, stream)

    def step(self, stream=None):
        for gs in self.groups:
            gs.step(stream)
        self.steps_done += 1
        if self.steps_done % self.period == 0:
            self.average(stream)
