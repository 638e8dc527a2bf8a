"""Conv -> BN -> SiLU blocks driven through the C ABI on one GPU.

Device memory comes from PyTorch (caching allocator) and every computation is a
call into ``libnumbat_conv.so``; this module only allocates buffers and orders the
calls: forward = conv_fwd (with fused batch statistics) then bn_silu_fwd; backward
= bn_silu_bwd, then conv_bwd_weight and conv_bwd_data.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

from . import numbat as nb

DEV = "cuda"


def dev_bf16(bits: np.ndarray, device=DEV) -> torch.Tensor:
    """Upload bf16 bit patterns (numpy uint16) as a bf16 tensor."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def dev_f32(a: np.ndarray, device=DEV) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


def host_f64(t: torch.Tensor) -> np.ndarray:
    """Exact widening of a bf16 / fp32 device tensor to float64 on the host."""
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def workspace(nbytes: int, device=DEV) -> Optional[torch.Tensor]:
    """A workspace for the C ABI: zero-filled (its leading counter header must start at zero)."""
    if nbytes == 0:
        return None
    return torch.zeros(nbytes, dtype=torch.uint8, device=device)


@dataclass
class ConvBlock:
    """One Conv+BN+SiLU layer: geometry, parameters and the buffers of one step."""

    n: int
    h: int
    w: int
    ci: int
    co: int
    k: int
    s: int
    eps: float = 1e-3
    momentum: float = 0.03
    x_pixel_stride: int = 0
    y_pixel_stride: int = 0
    bufs: dict = field(default_factory=dict)

    def __post_init__(self):
        self.p = self.k // 2
        self.prob = nb.conv_problem(self.n, self.h, self.w, self.ci, self.co, self.k, stride=self.s, pad=self.p,
                                    x_pixel_stride=self.x_pixel_stride, y_pixel_stride=self.y_pixel_stride)
        self.ho, self.wo = nb.numbat_conv_output_shape(self.prob)
        self.m = self.n * self.ho * self.wo
        self.ws_fwd = nb.numbat_workspace_size(nb.OP_CONV_FWD, self.prob)
        self.ws_dgrad = nb.numbat_workspace_size(nb.OP_CONV_BWD_DATA, self.prob)
        self.ws_wgrad = nb.numbat_workspace_size(nb.OP_CONV_BWD_WEIGHT, self.prob)

    def bn(self, a_pixel_stride=0, r_pixel_stride=0, dy_pixel_stride=0):
        return nb.bn_problem(self.m, self.co, self.eps, self.momentum, y_pixel_stride=self.y_pixel_stride,
                             a_pixel_stride=a_pixel_stride, r_pixel_stride=r_pixel_stride,
                             dy_pixel_stride=dy_pixel_stride)

    def ws_bytes(self) -> int:
        b = self.bn()
        return max(self.ws_fwd, self.ws_dgrad, self.ws_wgrad, nb.numbat_workspace_size(nb.OP_BN_SILU_FWD, b),
                   nb.numbat_workspace_size(nb.OP_BN_SILU_BWD, b))

    # ---- forward: y = conv(x, w) with fused stats, a = SiLU(BN(y)) [+ residual]
    def forward(self, x, w, gamma, beta, y=None, a=None, residual=None, ws=None, a_pixel_stride=0,
                r_pixel_stride=0, stream=None):
        y = y if y is not None else torch.empty((self.n, self.ho, self.wo, self.co), dtype=torch.bfloat16,
                                                  device=x.device)
        a = a if a is not None else torch.empty((self.n, self.ho, self.wo, self.co), dtype=torch.bfloat16,
                                                  device=x.device)
        ws = ws if ws is not None else workspace(self.ws_bytes(), x.device)
        stats = torch.empty(2 * self.co, dtype=torch.float32, device=x.device)
        save_mean = torch.empty(self.co, dtype=torch.float32, device=x.device)
        save_rstd = torch.empty(self.co, dtype=torch.float32, device=x.device)
        nb.numbat_conv_fwd(self.prob, x, w, y, stats, ws, stream=stream)
        nb.numbat_bn_silu_fwd(self.bn(a_pixel_stride, r_pixel_stride), y, stats, gamma, beta, residual, a, save_mean,
                              save_rstd, ws=ws, stream=stream)
        return {"y": y, "a": a, "stats": stats, "save_mean": save_mean, "save_rstd": save_rstd}

    # ---- backward
    def backward(self, g, x, w, gamma, beta, fwd, dx=None, accumulate_dx=False, residual_grad=None, ws=None,
                 g_pixel_stride=0, r_pixel_stride=0, want_dx=True, stream=None):
        dev = g.device
        ws = ws if ws is not None else workspace(self.ws_bytes(), dev)
        dy = torch.empty((self.n, self.ho, self.wo, self.co), dtype=torch.bfloat16, device=dev)
        dgamma = torch.empty(self.co, dtype=torch.float32, device=dev)
        dbeta = torch.empty(self.co, dtype=torch.float32, device=dev)
        nb.numbat_bn_silu_bwd(self.bn(g_pixel_stride, r_pixel_stride), g, fwd["y"], fwd["save_mean"],
                              fwd["save_rstd"], gamma, beta, dy, dgamma, dbeta, residual_grad, ws=ws, stream=stream)
        dw = torch.empty((self.co, self.k, self.k, self.ci), dtype=torch.float32, device=dev)
        nb.numbat_conv_bwd_weight(self.prob, x, dy, dw, False, ws, stream=stream)
        out = {"dy": dy, "dgamma": dgamma, "dbeta": dbeta, "dw": dw}
        if want_dx:
            if dx is None:
                dx = torch.empty((self.n, self.h, self.w, self.ci), dtype=torch.bfloat16, device=dev)
            nb.numbat_conv_bwd_data(self.prob, dy, w, dx, accumulate_dx, ws, stream=stream)
            out["dx"] = dx
        return out


class C2fBlock:
    """A C2f block (CSP backbone unit of the detector, Sec. 6.1) on the C ABI.

    cv1 (1x1, c1 -> c2), split into two c2/2 halves, nb bottlenecks of two 3x3 blocks with
    a residual add, concatenation of the 2 + nb halves, cv2 (1x1 -> c2).  Split and concat
    are zero-copy: every half lives at a channel offset of one concat buffer, read and
    written through pixel strides; the residual add is fused into the BN+SiLU forward, its
    gradient into the BN+SiLU backward (residual_grad), and the gradient fan-in of a half
    into the data-gradient accumulate flag.
    """

    def __init__(self, n, h, c1, c2, nb, eps=1e-3, shortcut=True):
        self.n, self.h, self.c1, self.c2, self.nb, self.eps, self.shortcut = n, h, c1, c2, nb, eps, shortcut
        self.half = c2 // 2
        self.catc = (2 + nb) * self.half
        hc = self.half
        self.cv1 = ConvBlock(n, h, h, c1, c2, 1, 1, eps=eps)
        self.m1 = ConvBlock(n, h, h, hc, hc, 3, 1, eps=eps, x_pixel_stride=self.catc)  # reads a half of cat
        self.m2 = ConvBlock(n, h, h, hc, hc, 3, 1, eps=eps)
        self.cv2 = ConvBlock(n, h, h, self.catc, c2, 1, 1, eps=eps)
        self.ws = workspace(max(b.ws_bytes() for b in (self.cv1, self.m1, self.m2, self.cv2)))

    def _half(self, t, k):
        return t[..., k * self.half:(k + 1) * self.half]

    def forward(self, x, params):
        """params: list of (w, gamma, beta) in order cv1, m0.cv1, m0.cv2, ..., cv2."""
        dev = x.device
        cat = torch.empty((self.n, self.h, self.h, self.catc), dtype=torch.bfloat16, device=dev)
        st = {"x": x, "cat": cat}
        w, g, b = params[0]
        st["cv1"] = self.cv1.forward(x, w, g, b, a=cat[..., :self.c2], ws=self.ws, a_pixel_stride=self.catc)
        for i in range(self.nb):
            inp = self._half(cat, 1 + i)
            w1, g1, b1 = params[1 + 2 * i]
            w2, g2, b2 = params[2 + 2 * i]
            f1 = self.m1.forward(inp, w1, g1, b1, ws=self.ws)
            f2 = self.m2.forward(f1["a"], w2, g2, b2, a=self._half(cat, 2 + i), ws=self.ws,
                                 residual=inp if self.shortcut else None, a_pixel_stride=self.catc,
                                 r_pixel_stride=self.catc)
            st[f"m{i}.cv1"], st[f"m{i}.cv2"] = f1, f2
        w, g, b = params[-1]
        st["cv2"] = self.cv2.forward(cat, w, g, b, ws=self.ws)
        st["out"] = st["cv2"]["a"]
        return st

    def backward(self, gout, st, params):
        """Returns (per-layer gradient dicts in params order, dx)."""
        grads = [None] * len(params)
        w, g, b = params[-1]
        grads[-1] = self.cv2.backward(gout, st["cat"], w, g, b, st["cv2"], ws=self.ws)
        dcat = grads[-1]["dx"]
        for i in reversed(range(self.nb)):
            gi = self._half(dcat, 2 + i)
            din = self._half(dcat, 1 + i)
            w1, g1, b1 = params[1 + 2 * i]
            w2, g2, b2 = params[2 + 2 * i]
            f1, f2 = st[f"m{i}.cv1"], st[f"m{i}.cv2"]
            b2g = self.m2.backward(gi, f1["a"], w2, g2, b2, f2, ws=self.ws, g_pixel_stride=self.catc,
                                   residual_grad=din if self.shortcut else None, r_pixel_stride=self.catc)
            b1g = self.m1.backward(b2g["dx"], self._half(st["cat"], 1 + i), w1, g1, b1, f1, dx=din,
                                   accumulate_dx=True, ws=self.ws)
            grads[1 + 2 * i], grads[2 + 2 * i] = b1g, b2g
        w, g, b = params[0]
        grads[0] = self.cv1.backward(dcat[..., :self.c2], st["x"], w, g, b, st["cv1"], ws=self.ws,
                                     g_pixel_stride=self.catc)
        return grads, grads[0]["dx"]


class DetectHeadInfer:
    """One scale of the architecture-faithful decoupled detect head (Sec. 6.1) in inference
    mode on the C ABI: a box branch (3x3 c -> 64, 3x3 64 -> 64, 1x1 64 -> 64 + bias) and a
    class branch (3x3 c -> 192, 3x3 192 -> 192, 1x1 192 -> 80 + bias).  Each 3x3 layer is one
    numbat_conv_bn_silu_infer call (BN with running statistics folded into the conv's output
    stage); the two 1x1 prediction convs write channel slices 0..63 and 64..143 of one
    [n, h, w, 144] output (zero-copy concatenation)."""

    BOX, CLS, NCLS, REG = 64, 192, 80, 64

    def __init__(self, n, h, c, eps=1e-3):
        self.n, self.h, self.c, self.eps = n, h, c, eps
        self.out_c = self.REG + self.NCLS
        self.p3 = {co_ci: nb.conv_problem(n, h, h, co_ci[1], co_ci[0], 3) for co_ci in
                   ((self.BOX, c), (self.BOX, self.BOX), (self.CLS, c), (self.CLS, self.CLS))}
        self.p_box = nb.conv_problem(n, h, h, self.BOX, self.REG, 1, y_pixel_stride=self.out_c)
        self.p_cls = nb.conv_problem(n, h, h, self.CLS, self.NCLS, 1, y_pixel_stride=self.out_c)

    def forward(self, x, box, cls, stream=None):
        """box / cls: [(w, gamma, beta, mean, var), (w, gamma, beta, mean, var), (w, bias)]."""
        dev = x.device
        out = torch.empty((self.n, self.h, self.h, self.out_c), dtype=torch.bfloat16, device=dev)
        for layers, width, dst, p1 in ((box, self.BOX, out[..., :self.REG], self.p_box),
                                       (cls, self.CLS, out[..., self.REG:], self.p_cls)):
            a = x
            for (w, g, b, m, v), ci in zip(layers[:2], (self.c, width)):
                y = torch.empty((self.n, self.h, self.h, width), dtype=torch.bfloat16, device=dev)
                nb.numbat_conv_bn_silu_infer(self.p3[(width, ci)], a, w, g, b, m, v, self.eps, y, stream=stream)
                a = y
            w, bias = layers[2]
            nb.numbat_conv_fwd_bias(p1, a, w, bias, dst, stream=stream)
        return out
