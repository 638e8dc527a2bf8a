"""The detector's backbone and neck as one network on the C ABI (chain mode): the 65
Conv+BN+SiLU layers of the workload table connected as the case study's network (Sec. 6.1:
CSP backbone of C2f blocks and an SPPF block, PAN-FPN neck with nearest upsampling and
concatenations), forward and backward.  The backward runs each layer's weight gradient on
a second stream (nothing later in the backward reads it), each enqueued after the next
layer's BN backward behind a wait for its own data gradient, as the conv-set schedule does.

Every concatenation is a buffer whose channel slices the producers write and the consumers
read through pixel strides (no copies): a C2f block's halves live in its own concat buffer,
an SPPF's pooled maps in its concat buffer, and a tensor that feeds a neck concatenation is
written straight into that concatenation's slice.  Gradients mirror the activations: each
gradient buffer is written by its first producer in the backward and accumulated into by
the second (data-gradient `accumulate`, BN backward `residual_grad` for the bottleneck
residuals, upsample/max-pool backward `accumulate`).  Device memory comes from PyTorch; every
computation is a call into the HIP library.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np
import torch

from . import blocks, synth, workloads
from . import numbat as nb

BF = torch.bfloat16
C2F = {"b2": (2, True), "b4": (4, True), "b6": (4, True), "b8": (2, True),
       "n12": (2, False), "n15": (2, False), "n18": (2, False), "n21": (2, False)}


class Conv:
    """One Conv+BN+SiLU layer: descriptors, its own buffers, and views into shared ones."""

    def __init__(self, spec, n, h, eps, x, dx, out, dout, x_stride=0, out_stride=0, res=None, dres=None,
                 res_stride=0):
        self.name, self.spec = spec.name, spec
        self.blk = blocks.ConvBlock(n, h, h, spec.ci, spec.co, spec.k, spec.s, eps=eps, x_pixel_stride=x_stride)
        ho = self.blk.ho
        dev = "cuda"
        self.x, self.dx, self.out, self.dout = x, dx, out, dout
        self.res, self.dres = res, dres
        self.bnp = self.blk.bn(a_pixel_stride=out_stride, r_pixel_stride=res_stride)
        self.y = torch.empty((n, ho, ho, spec.co), dtype=BF, device=dev)
        self.dy = torch.empty_like(self.y)
        f32 = lambda k: torch.empty(k, dtype=torch.float32, device=dev)
        self.stats, self.smean, self.srstd = f32(2 * spec.co), f32(spec.co), f32(spec.co)
        self.dgamma, self.dbeta = f32(spec.co), f32(spec.co)
        self.dw = torch.empty((spec.co, spec.k, spec.k, spec.ci), dtype=torch.float32, device=dev)
        self.acc_dx = False  # set by the network: does this layer's dx add to an earlier gradient?

    def fwd(self, w, g, b, ws):
        nb.numbat_conv_fwd(self.blk.prob, self.x, w, self.y, self.stats, ws)
        nb.numbat_bn_silu_fwd(self.bnp, self.y, self.stats, g, b, self.res, self.out, self.smean, self.srstd, ws=ws)

    def bwd(self, w, g, b, ws, want_dx=True, side=None, ws_side=None, pending=None):
        """BN/SiLU backward, then the data and weight gradients.  With a side stream, returns
        a callable that enqueues the weight gradient there (on ws_side) after a wait for this
        layer's data gradient (`.done`); `pending`, if given, runs between the BN backward and
        the data gradient to enqueue earlier layers' weight gradients."""
        nb.numbat_bn_silu_bwd(self.bnp, self.dout, self.y, self.smean, self.srstd, g, b, self.dy, self.dgamma,
                              self.dbeta, self.dres, ws=ws)
        if side is None:
            nb.numbat_conv_bwd_weight(self.blk.prob, self.x, self.dy, self.dw, False, ws)
            if want_dx:
                nb.numbat_conv_bwd_data(self.blk.prob, self.dy, w, self.dx, self.acc_dx, ws)
            return None
        if pending is not None:
            pending()
        if want_dx:
            nb.numbat_conv_bwd_data(self.blk.prob, self.dy, w, self.dx, self.acc_dx, ws)
        done = torch.cuda.Event()
        done.record()

        def wgrad(wait=True):
            if wait:
                side.wait_event(done)
            with torch.cuda.stream(side):
                nb.numbat_conv_bwd_weight(self.blk.prob, self.x, self.dy, self.dw, False, ws_side)

        wgrad.done = done
        return wgrad


class Detector:
    """Backbone + neck at batch n and a square input of side hin (a multiple of 32)."""

    def __init__(self, n: int, hin: int, eps: float = 1e-3):
        assert hin % 32 == 0
        self.n, self.hin, self.eps = n, hin, eps
        self.specs = {l.name: l for l in workloads.backbone_neck_layers()}
        dev = "cuda"
        buf = lambda h, c: torch.empty((n, h, h, c), dtype=BF, device=dev)
        S = {k: hin >> k for k in range(1, 6)}  # side at stride 2^k
        self.layers: List[Conv] = []
        self.ops: List[Tuple] = []  # forward program: ("conv", Conv) / ("pool", ...) / ("up", ...)
        L = {}

        def conv(name, h, x, dx, out, dout, **kw):
            c = Conv(self.specs[name], n, h, eps, x, dx, out, dout, **kw)
            L[name] = c
            self.layers.append(c)
            self.ops.append(("conv", c))
            return c

        def c2f(prefix, h, x, dx, out, dout, x_stride=0, out_stride=0):
            nbk, sc = C2F[prefix]
            c1, c2 = self.specs[prefix + ".cv1"].ci, self.specs[prefix + ".cv1"].co
            half = c2 // 2
            catc = (2 + nbk) * half
            cat, dcat = buf(h, catc), buf(h, catc)
            sl = lambda t, k: t[..., k * half:(k + 1) * half]
            conv(prefix + ".cv1", h, x, dx, cat[..., :c2], dcat[..., :c2], x_stride=x_stride, out_stride=catc)
            for i in range(nbk):
                tmp, dtmp = buf(h, half), buf(h, half)
                conv(f"{prefix}.m{i}.cv1", h, sl(cat, 1 + i), sl(dcat, 1 + i), tmp, dtmp, x_stride=catc)
                conv(f"{prefix}.m{i}.cv2", h, tmp, dtmp, sl(cat, 2 + i), sl(dcat, 2 + i), out_stride=catc,
                     res=sl(cat, 1 + i) if sc else None, dres=sl(dcat, 1 + i) if sc else None,
                     res_stride=catc if sc else 0)
                L[f"{prefix}.m{i}.cv1"].acc_dx = True  # adds to the half's gradient (cv1 / residual)
            conv(prefix + ".cv2", h, cat, dcat, out, dout, out_stride=out_stride)

        self.x, self.dx = buf(hin, 3), buf(hin, 3)
        a0, da0 = buf(S[1], 48), buf(S[1], 48)
        a1, da1 = buf(S[2], 96), buf(S[2], 96)
        a2, da2 = buf(S[2], 96), buf(S[2], 96)
        a3, da3 = buf(S[3], 192), buf(S[3], 192)
        n14, dn14 = buf(S[3], 576), buf(S[3], 576)      # [up(a12) | a4]
        a5, da5 = buf(S[4], 384), buf(S[4], 384)
        n11, dn11 = buf(S[4], 960), buf(S[4], 960)      # [up(a9) | a6]
        a7, da7 = buf(S[5], 576), buf(S[5], 576)
        a8, da8 = buf(S[5], 576), buf(S[5], 576)
        sp, dsp = buf(S[5], 1152), buf(S[5], 1152)      # SPPF [s | m1 | m2 | m3]
        n20, dn20 = buf(S[5], 960), buf(S[5], 960)      # [a19 | a9]
        n17, dn17 = buf(S[4], 576), buf(S[4], 576)      # [a16 | a12]
        self.p3, self.g3 = buf(S[3], 192), buf(S[3], 192)
        self.p4, self.g4 = buf(S[4], 384), buf(S[4], 384)
        self.p5, self.g5 = buf(S[5], 576), buf(S[5], 576)

        conv("b0", hin, self.x, self.dx, a0, da0)
        conv("b1", S[1], a0, da0, a1, da1)
        c2f("b2", S[2], a1, da1, a2, da2)
        conv("b3", S[2], a2, da2, a3, da3)
        c2f("b4", S[3], a3, da3, n14[..., 384:], dn14[..., 384:], out_stride=576)
        conv("b5", S[3], n14[..., 384:], dn14[..., 384:], a5, da5, x_stride=576)
        L["b5"].acc_dx = True   # adds to n15's gradient of a4
        c2f("b6", S[4], a5, da5, n11[..., 576:], dn11[..., 576:], out_stride=960)
        conv("b7", S[4], n11[..., 576:], dn11[..., 576:], a7, da7, x_stride=960)
        L["b7"].acc_dx = True   # adds to n12's gradient of a6
        c2f("b8", S[5], a7, da7, a8, da8)
        conv("b9.cv1", S[5], a8, da8, sp[..., :288], dsp[..., :288], out_stride=1152)
        pp = nb.pool_problem(n, S[5], S[5], 288, 1152, 1152)
        self.idx = [torch.empty((n, S[5], S[5], 288), dtype=torch.uint8, device=dev) for _ in range(3)]
        for k in range(3):
            self.ops.append(("pool", pp, sp[..., 288 * k:288 * (k + 1)], sp[..., 288 * (k + 1):288 * (k + 2)],
                             self.idx[k], dsp[..., 288 * (k + 1):288 * (k + 2)], dsp[..., 288 * k:288 * (k + 1)]))
        conv("b9.cv2", S[5], sp, dsp, n20[..., 384:], dn20[..., 384:], out_stride=960)
        self.ops.append(("up", nb.pool_problem(n, S[5], S[5], 576, 960, 960), n20[..., 384:], n11[..., :576],
                         dn11[..., :576], dn20[..., 384:]))
        c2f("n12", S[4], n11, dn11, n17[..., 192:], dn17[..., 192:], out_stride=576)
        self.ops.append(("up", nb.pool_problem(n, S[4], S[4], 384, 576, 576), n17[..., 192:], n14[..., :384],
                         dn14[..., :384], dn17[..., 192:]))
        c2f("n15", S[3], n14, dn14, self.p3, self.g3)
        conv("n16", S[3], self.p3, self.g3, n17[..., :192], dn17[..., :192], out_stride=576)
        L["n16"].acc_dx = True  # adds to P3's upstream gradient
        c2f("n18", S[4], n17, dn17, self.p4, self.g4)
        conv("n19", S[4], self.p4, self.g4, n20[..., :384], dn20[..., :384], out_stride=960)
        L["n19"].acc_dx = True  # adds to P4's upstream gradient
        c2f("n21", S[5], n20, dn20, self.p5, self.g5)
        self.L = L
        self.ws = torch.zeros(max(c.blk.ws_bytes() for c in self.layers), dtype=torch.uint8, device=dev)
        self.ws_side = torch.zeros_like(self.ws)
        self.side = torch.cuda.Stream()  # default priority
        self.flops = 3 * sum(self.specs[c.name].gemm_flops(n) * (hin / 640.0) ** 2 for c in self.layers)

    # ---- parameters and inputs
    def seeded(self, cfg_index: int, g_std: float = 1.0, affine: bool = False):
        """Seeded parameters (Kaiming-uniform weights; gamma 1, beta 0, or seeded affine
        ones) and inputs: an image-like input in [0, 1) and N(0, g_std) upstream gradients of
        P3, P4, P5.  Returns the host bf16/fp32 arrays for the oracle."""
        host = {}
        names = [l.name for l in workloads.backbone_neck_layers()]
        self.params = {}
        for i, name in enumerate(names):
            sp = self.specs[name]
            sid = lambda t: synth.stream_id(cfg_index, i, t)
            b = synth.kaiming_uniform_bound(sp.ci * sp.k * sp.k)
            w = synth.bf16((sp.co, sp.k, sp.k, sp.ci), sid(synth.T_W), synth.UNIFORM, -b, b)
            if affine:
                g = synth.f32((sp.co,), sid(synth.T_GAMMA), synth.UNIFORM, 0.5, 1.5)
                be = synth.f32((sp.co,), sid(synth.T_BETA), synth.NORMAL, 0.0, 0.1)
            else:
                g, be = np.ones(sp.co, np.float32), np.zeros(sp.co, np.float32)
            host[name] = (w, g, be)
            self.params[name] = (blocks.dev_bf16(w), blocks.dev_f32(g), blocks.dev_f32(be))
        sid = lambda t: synth.stream_id(cfg_index, 999, t)
        xb = synth.bf16(tuple(self.x.shape), sid(synth.T_X), synth.UNIFORM, 0.0, 1.0)
        self.x.copy_(blocks.dev_bf16(xb))
        gs = []
        for k, t in enumerate((self.g3, self.g4, self.g5)):
            gb = synth.bf16(tuple(t.shape), synth.stream_id(cfg_index, 1000 + k, synth.T_G), synth.NORMAL, 0.0, g_std)
            gs.append(gb)
        self.g_init = [blocks.dev_bf16(gb) for gb in gs]
        return host, xb, gs

    # ---- one training step
    def forward(self):
        for op in self.ops:
            if op[0] == "conv":
                c = op[1]
                c.fwd(*self.params[c.name], self.ws)
            elif op[0] == "pool":
                _, pp, src, dst, idx, _, _ = op
                nb.numbat_maxpool5_fwd(pp, src, dst, idx)
            else:
                _, pp, src, dst, _, _ = op
                nb.numbat_upsample2x_fwd(pp, src, dst)

    def backward(self, overlap=True, group=1, tail=0):
        """The backward in reverse program order.  overlap=False keeps everything on the
        current stream; otherwise the weight gradients run on the side stream in groups of
        `group` layers behind one wait (the last `tail` convs of the backward one by one)."""
        # the outputs' upstream gradients (P3 and P4 also receive the stride-2 convs' dx)
        for t, g in zip((self.g3, self.g4, self.g5), self.g_init):
            t.copy_(g)
        sd = self.side if overlap else None
        if sd is not None:
            sd.wait_stream(torch.cuda.current_stream())
        queued = []

        def flush():
            if queued:
                sd.wait_event(queued[-1].done)
            for f in queued:
                f(wait=False)
            queued.clear()

        nconv = len(self.layers)
        i = 0
        for op in reversed(self.ops):
            if op[0] == "conv":
                c = op[1]
                gsz = 1 if i >= nconv - tail else group
                i += 1
                r = c.bwd(*self.params[c.name], self.ws, want_dx=True, side=sd, ws_side=self.ws_side,
                          pending=flush if len(queued) >= gsz else None)
                if r is not None:
                    queued.append(r)
            elif op[0] == "pool":
                _, pp, _, _, idx, ddst, dsrc = op
                nb.numbat_maxpool5_bwd(pp, ddst, idx, dsrc, True)
            else:
                _, pp, _, _, ddst, dsrc = op
                nb.numbat_upsample2x_bwd(pp, ddst, dsrc, True)
        if sd is not None:
            flush()
            # the next forward overwrites the activations the weight gradients read
            torch.cuda.current_stream().wait_stream(sd)

    def step(self, overlap=True):
        self.forward()
        self.backward(overlap)
