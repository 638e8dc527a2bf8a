"""The training-step schedule of a conv set on one GPU: buffers of every layer and the
order in which the C-ABI calls are enqueued.

One step = every layer's forward in network order (conv_fwd with fused batch statistics,
then bn_silu_fwd), then the backward in reverse order (bn_silu_bwd, conv_bwd_data,
conv_bwd_weight).  With `fuse_bwd` (off by default: slower on this GPU), a layer whose data
gradient takes the BN + SiLU backward prologue (the 3x3 stride-1 layers) runs bn_silu_bwd
for dgamma and dbeta only and then numbat_conv_bwd_data_bn_silu_prologue, which forms dy
inside the data gradient and writes it for the weight gradient; the results are the same
bit for bit.  Two schedules
give the same results bit for bit (every kernel and every reduction order is the same;
only the streams differ):

* serial: everything on the current stream;
* two streams: each layer's weight gradient (which nothing later in the backward reads)
  runs on a second stream with its own workspace, after that layer's data gradient.  The
  weight gradients are enqueued in groups behind one cross-stream wait (each wait costs the
  main queue a completion signal), and a group is enqueued after the next layer's BN
  backward: in a captured graph a data gradient's first dependant is then the next
  main-stream kernel, which keeps the main chain on one hardware queue.

Device memory comes from PyTorch; every computation is a call into the HIP library.
"""
from __future__ import annotations

import torch

from . import blocks, synth
from . import numbat as nb


class Layer:
    """Device buffers, seeded inputs and problem descriptors of one layer of a conv set."""

    def __init__(self, idx, spec, n, cfg_index, eps, g_std=1.0, fuse_bwd=False):
        self.spec = spec
        self.name = spec.name
        sid = lambda t: synth.stream_id(cfg_index, idx, t)
        b = synth.kaiming_uniform_bound(spec.ci * spec.k * spec.k)
        self.blk = blocks.ConvBlock(n, spec.h, spec.h, spec.ci, spec.co, spec.k, spec.s, eps=eps)
        ho = self.blk.ho
        self.x = blocks.dev_bf16(synth.bf16((n, spec.h, spec.h, spec.ci), sid(synth.T_X)))
        self.w = blocks.dev_bf16(synth.bf16((spec.co, spec.k, spec.k, spec.ci), sid(synth.T_W), synth.UNIFORM, -b, b))
        self.g = blocks.dev_bf16(synth.bf16((n, ho, ho, spec.co), sid(synth.T_G), synth.NORMAL, 0.0, g_std))
        dev = self.x.device
        bf = torch.bfloat16
        self.gamma = torch.ones(spec.co, device=dev)
        self.beta = torch.zeros(spec.co, device=dev)
        self.y = torch.empty((n, ho, ho, spec.co), dtype=bf, device=dev)
        self.a = torch.empty_like(self.y)
        self.dy = torch.empty_like(self.y)
        self.dx = torch.empty((n, spec.h, spec.h, spec.ci), dtype=bf, device=dev)
        self.dw = torch.empty((spec.co, spec.k, spec.k, spec.ci), dtype=torch.float32, device=dev)
        f32 = lambda k: torch.empty(k, dtype=torch.float32, device=dev)
        self.stats, self.smean, self.srstd, self.dgamma, self.dbeta = (f32(2 * spec.co), f32(spec.co),
                                                                       f32(spec.co), f32(spec.co), f32(spec.co))
        self.bnp = self.blk.bn()
        self.ws_need = self.blk.ws_bytes()
        self.fused = fuse_bwd and self._prologue_supported()
        self.flops = spec.gemm_flops(n)  # one pass
        self.bn_elems = self.blk.m * spec.co

    def _prologue_supported(self):
        try:
            nb.numbat_workspace_size(nb.OP_CONV_BWD_DATA_BN_SILU, self.blk.prob)
        except nb.NumbatError as e:
            if e.status == nb.ERR_UNSUPPORTED:
                return False
            raise
        return True

    def _bn_bwd(self):
        """BN + SiLU backward: dgamma, dbeta (and dy unless the data gradient forms it)"""
        nb.numbat_bn_silu_bwd(self.bnp, self.g, self.y, self.smean, self.srstd, self.gamma, self.beta,
                              None if self.fused else self.dy, self.dgamma, self.dbeta, None, ws=self.ws,
                              ws_bytes=self.ws_len)

    def _dgrad(self):
        if self.fused:
            nb.numbat_conv_bwd_data_bn_silu_prologue(self.blk.prob, self.g, self.y, self.smean, self.srstd, self.gamma,
                                                     self.beta, self.dgamma, self.dbeta, self.w, self.dx, self.dy)
        else:
            nb.numbat_conv_bwd_data(self.blk.prob, self.dy, self.w, self.dx, False, self.ws, ws_bytes=self.ws_len)

    def outputs(self):
        """Every tensor one step writes, by name."""
        return {"y": self.y, "a": self.a, "stats": self.stats, "save_mean": self.smean, "save_rstd": self.srstd,
                "dy": self.dy, "dgamma": self.dgamma, "dbeta": self.dbeta, "dx": self.dx, "dw": self.dw}

    def bind_ws(self, ws, ws_side):
        self.ws, self.ws_side = ws, ws_side
        self.ws_len = ws.numel()

    def fwd(self, ev=None):
        e = ev.get(self.name) if ev else None
        if e: e[0].record()
        nb.numbat_conv_fwd(self.blk.prob, self.x, self.w, self.y, self.stats, self.ws, ws_bytes=self.ws_len)
        if e: e[1].record()
        nb.numbat_bn_silu_fwd(self.bnp, self.y, self.stats, self.gamma, self.beta, None, self.a, self.smean,
                              self.srstd, ws=self.ws, ws_bytes=self.ws_len)
        if e: e[2].record()

    def bwd(self, ev=None, side=None, pending=None, defer=True):
        """BN/SiLU backward, then the data and weight gradients.  With a side stream the
        weight gradient runs there, on its own workspace.  With `defer`, this returns a
        callable that enqueues this layer's weight gradient (by default after a wait for
        this layer's data gradient; `.done` is that event), and `pending`, if given, runs
        between this layer's BN backward and its data gradient to enqueue earlier layers'
        weight gradients."""
        e = ev.get(self.name) if ev else None
        if e: e[3].record()
        self._bn_bwd()
        if e: e[4].record()
        if side is not None:
            if pending is not None:
                pending()
            self._dgrad()
            done = torch.cuda.Event()
            done.record()

            def wgrad(wait=True):
                if wait:
                    side.wait_event(done)
                with torch.cuda.stream(side):
                    nb.numbat_conv_bwd_weight(self.blk.prob, self.x, self.dy, self.dw, False, self.ws_side,
                                              ws_bytes=self.ws_len)

            wgrad.done = done
            if defer:
                return wgrad
            wgrad()
            return None
        # serial: the weight gradient, then the data gradient (events 4-5, 5-6); a fused layer
        # forms dy in its data gradient, which then comes first (events 4-5 data, 5-6 weight)
        if self.fused:
            self._dgrad()
            if e: e[5].record()
            nb.numbat_conv_bwd_weight(self.blk.prob, self.x, self.dy, self.dw, False, self.ws, ws_bytes=self.ws_len)
            if e: e[6].record()
            return None
        nb.numbat_conv_bwd_weight(self.blk.prob, self.x, self.dy, self.dw, False, self.ws, ws_bytes=self.ws_len)
        if e: e[5].record()
        self._dgrad()
        if e: e[6].record()


class ConvSet:
    """Every layer of a conv set with shared workspaces, and the step over them."""

    def __init__(self, specs, n, cfg_index, eps, g_std=1.0, layer_index=None, fuse_bwd=False):
        idx = layer_index or list(range(len(specs)))
        self.layers = [Layer(i, l, n, cfg_index, eps, g_std, fuse_bwd) for i, l in zip(idx, specs)]
        need = max(l.ws_need for l in self.layers)
        self.ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
        self.ws_side = torch.zeros_like(self.ws)
        for l in self.layers:
            l.bind_ws(self.ws, self.ws_side)
        self.side = torch.cuda.Stream()  # default priority

    def step(self, ev=None, overlap=True, defer=True, group=1, tail=0):
        """One training step: every layer's forward, then the backward in reverse order.
        overlap=False keeps everything on the current stream; otherwise the weight gradients
        run on the side stream (`defer`: in groups of `group` layers behind one wait, the
        last `tail` layers of the backward one by one; else each right after its data
        gradient)."""
        sd = self.side if overlap else None
        for l in self.layers:
            l.fwd(ev)
        queued = []  # weight gradients not yet enqueued; the last one's wait covers all

        def flush():
            if queued:
                self.side.wait_event(queued[-1].done)
            for f in queued:
                f(wait=False)
            queued.clear()

        nl = len(self.layers)
        for i, l in enumerate(reversed(self.layers)):
            g = 1 if i >= nl - tail else group
            r = l.bwd(ev, sd, flush if len(queued) >= g else None, defer)
            if r is not None:
                queued.append(r)
        flush()
        if sd is not None:
            torch.cuda.current_stream().wait_stream(sd)
