"""ORACLE -- test infrastructure only.  The architecture-faithful decoupled detect head in
inference mode, float64 (Sec. 6.1: decoupled head at strides 8/16/32; Table 2 #9: evaluation
with running BN statistics).

Per scale (input feature map of C channels): a box branch Conv3x3(C->64)+BN+SiLU,
Conv3x3(64->64)+BN+SiLU, Conv1x1(64->64)+bias, and a class branch Conv3x3(C->192)+BN+SiLU,
Conv3x3(192->192)+BN+SiLU, Conv1x1(192->80)+bias; the two outputs are concatenated along
channels (box first) into [N, H, W, 144].  BN uses running statistics.
"""
from __future__ import annotations

import numpy as np

from . import ConvShape, bn_silu_eval, conv_fwd, conv_fwd_bias


def branch(x, layers, eps):
    """layers: list of dicts with w, and either (gamma, beta, mean, var) or bias."""
    a = np.asarray(x, np.float64)
    for L in layers:
        n, h, w_, c = a.shape
        co, k = L["w"].shape[0], L["w"].shape[1]
        s = ConvShape(n, h, w_, c, co, k, k, 1, 1, k // 2, k // 2)
        if "bias" in L:
            a = conv_fwd_bias(a, L["w"], L["bias"], s)
        else:
            a = bn_silu_eval(conv_fwd(a, L["w"], s), L["mean"], L["var"], L["gamma"], L["beta"], eps)
    return a


def head_infer(x, box_layers, cls_layers, eps):
    """[N, H, W, 64 + 80]: box branch output, then class branch output."""
    return np.concatenate([branch(x, box_layers, eps), branch(x, cls_layers, eps)], axis=-1)
