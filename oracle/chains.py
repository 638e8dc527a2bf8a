"""ORACLE -- test infrastructure only.  Multi-block dataflow of the detector, float64.

Composes the single-block oracle (``oracle.block_fwd`` / ``block_bwd``) into the
chains the case study's network is made of (Sec. 6.1: CSP backbone of C2f
blocks):
  * ``chain_fwd`` / ``chain_bwd``: blocks applied one after another (the stem);
  * ``c2f_fwd`` / ``c2f_bwd``: a C2f block -- 1x1 conv, split into two halves,
    n bottlenecks each of two 3x3 Conv+BN+SiLU blocks with a residual add,
    concatenation of all halves, 1x1 conv.
Backward passes follow the chain rule through split (gradient of a slice),
concat (gradients scattered back to slices) and residual add (gradient passes
to both operands unchanged).
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from . import ConvShape, block_bwd, block_fwd


def chain_fwd(x, ws: Sequence[np.ndarray], shapes: Sequence[ConvShape], gammas, betas, eps):
    acts = [np.asarray(x, np.float64)]
    fwds = []
    for w, s, g, b in zip(ws, shapes, gammas, betas):
        f = block_fwd(acts[-1], w, s, g, b, eps)
        fwds.append(f)
        acts.append(f["a"])
    return acts, fwds


def chain_bwd(g, acts, fwds, ws, shapes, gammas, betas, eps):
    grads: List[Dict] = [None] * len(ws)
    up = np.asarray(g, np.float64)
    for i in reversed(range(len(ws))):
        grads[i] = block_bwd(up, acts[i], ws[i], shapes[i], fwds[i], gammas[i], betas[i], eps)
        up = grads[i]["dx"]
    return grads, up


def c2f_shapes(n: int, h: int, c1: int, c2: int, nb: int):
    half = c2 // 2
    cv1 = ConvShape(n, h, h, c1, c2, 1, 1)
    m = ConvShape(n, h, h, half, half, 3, 3, 1, 1, 1, 1)
    cv2 = ConvShape(n, h, h, (2 + nb) * half, c2, 1, 1)
    return cv1, m, cv2


def c2f_fwd(x, params, n: int, h: int, c1: int, c2: int, nb: int, eps, shortcut=True):
    """params: list of (w, gamma, beta) in order cv1, m0.cv1, m0.cv2, ..., cv2."""
    cv1, m, cv2 = c2f_shapes(n, h, c1, c2, nb)
    half = c2 // 2
    st = {"x": np.asarray(x, np.float64)}
    w, g, b = params[0]
    st["cv1"] = block_fwd(st["x"], w, cv1, g, b, eps)
    pieces = [st["cv1"]["a"][..., :half], st["cv1"]["a"][..., half:]]
    for i in range(nb):
        inp = pieces[-1]
        w1, g1, b1 = params[1 + 2 * i]
        w2, g2, b2 = params[2 + 2 * i]
        f1 = block_fwd(inp, w1, m, g1, b1, eps)
        f2 = block_fwd(f1["a"], w2, m, g2, b2, eps, residual=inp if shortcut else None)
        st[f"m{i}.in"] = inp
        st[f"m{i}.cv1"] = f1
        st[f"m{i}.cv2"] = f2
        pieces.append(f2["a"])
    st["cat"] = np.concatenate(pieces, axis=-1)
    w, g, b = params[-1]
    st["cv2"] = block_fwd(st["cat"], w, cv2, g, b, eps)
    st["out"] = st["cv2"]["a"]
    return st


def c2f_bwd(gout, st, params, n: int, h: int, c1: int, c2: int, nb: int, eps, shortcut=True):
    """Returns (grads per parameter block in params order, dx)."""
    cv1, m, cv2 = c2f_shapes(n, h, c1, c2, nb)
    half = c2 // 2
    grads = [None] * len(params)
    w, g, b = params[-1]
    grads[-1] = block_bwd(gout, st["cat"], w, cv2, st["cv2"], g, b, eps)
    dcat = grads[-1]["dx"]
    dpieces = [dcat[..., k * half:(k + 1) * half].copy() for k in range(2 + nb)]
    for i in reversed(range(nb)):
        gi = dpieces[2 + i]
        w1, g1, b1 = params[1 + 2 * i]
        w2, g2, b2 = params[2 + 2 * i]
        b2g = block_bwd(gi, st[f"m{i}.cv1"]["a"], w2, m, st[f"m{i}.cv2"], g2, b2, eps)
        b1g = block_bwd(b2g["dx"], st[f"m{i}.in"], w1, m, st[f"m{i}.cv1"], g1, b1, eps)
        grads[1 + 2 * i] = b1g
        grads[2 + 2 * i] = b2g
        dpieces[1 + i] = dpieces[1 + i] + b1g["dx"] + (gi if shortcut else 0.0)
    dcv1 = np.concatenate(dpieces[:2], axis=-1)
    w, g, b = params[0]
    grads[0] = block_bwd(dcv1, st["x"], w, cv1, st["cv1"], g, b, eps)
    return grads, grads[0]["dx"]
