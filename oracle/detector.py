"""ORACLE -- test infrastructure only.  The detector's backbone and neck as one network
(chain mode), float64: the real dataflow between the 65 Conv+BN+SiLU layers of the
workload table (Sec. 6.1: CSP backbone of C2f blocks with an SPPF block, PAN-FPN neck with
nearest upsampling and concatenations), forward and backward.

Forward (a_k: activation of stage k; cat: channel concatenation, first operand first):
  a0 = conv b0 (s2), a1 = conv b1 (s2), a2 = C2f b2 (residual), a3 = conv b3 (s2),
  a4 = C2f b4 (residual), a5 = conv b5 (s2), a6 = C2f b6 (residual), a7 = conv b7 (s2),
  a8 = C2f b8 (residual),
  SPPF: s = conv b9.cv1, m1 = pool(s), m2 = pool(m1), m3 = pool(m2), a9 = conv b9.cv2(cat[s, m1, m2, m3]),
  a12 = C2f n12(cat[up(a9), a6]),  a15 = C2f n15(cat[up(a12), a4])          -> P3 = a15
  a18 = C2f n18(cat[conv n16 (s2) of a15, a12])                              -> P4 = a18
  a21 = C2f n21(cat[conv n19 (s2) of a18, a9])                               -> P5 = a21
(neck C2f blocks have no residual; pool is the 5x5 stride-1 max pool, up the nearest 2x).
The backward takes upstream gradients of P3, P4, P5 and follows the chain rule in reverse;
a tensor consumed twice receives the sum of both gradients.
"""
from __future__ import annotations

import numpy as np

from . import ConvShape, block_bwd, block_fwd
from .chains import c2f_bwd, c2f_fwd
from .pool import maxpool_bwd, maxpool_fwd, upsample2x_bwd, upsample2x_fwd

C2F = {"b2": (2, True), "b4": (4, True), "b6": (4, True), "b8": (2, True),
       "n12": (2, False), "n15": (2, False), "n18": (2, False), "n21": (2, False)}


def _conv(name, x, P, eps, stride):
    n, h, w, c = x.shape
    wt = P[name][0]
    k = wt.shape[1]
    s = ConvShape(n, h, w, c, wt.shape[0], k, k, stride, stride, k // 2, k // 2)
    return s, block_fwd(x, wt, s, P[name][1], P[name][2], eps)


def _c2f_params(prefix, P):
    nb = C2F[prefix][0]
    names = [f"{prefix}.cv1"] + [f"{prefix}.m{i}.cv{j}" for i in range(nb) for j in (1, 2)] + [f"{prefix}.cv2"]
    return names, [P[nm] for nm in names]


def _c2f(prefix, x, P, eps):
    nb, sc = C2F[prefix]
    names, params = _c2f_params(prefix, P)
    n, h, _, c1 = x.shape
    c2 = params[-1][0].shape[0]
    return c2f_fwd(x, params, n, h, c1, c2, nb, eps, sc)


def forward(x, P, eps):
    """P: layer name -> (w, gamma, beta).  Returns the state the backward needs; st['P3'],
    st['P4'], st['P5'] are the outputs."""
    st = {"x": np.asarray(x, np.float64)}
    a = st["x"]
    for name, kind in (("b0", "s2"), ("b1", "s2"), ("b2", "c2f"), ("b3", "s2"), ("b4", "c2f"), ("b5", "s2"),
                       ("b6", "c2f"), ("b7", "s2"), ("b8", "c2f")):
        st[name + ".in"] = a
        if kind == "s2":
            st[name + ".shape"], st[name] = _conv(name, a, P, eps, 2)
            a = st[name]["a"]
        else:
            st[name] = _c2f(name, a, P, eps)
            a = st[name]["out"]
    st["b9.in"] = a
    st["b9.cv1.shape"], st["b9.cv1"] = _conv("b9.cv1", a, P, eps, 1)
    s1 = st["b9.cv1"]["a"]
    m1, i1 = maxpool_fwd(s1)
    m2, i2 = maxpool_fwd(m1)
    m3, i3 = maxpool_fwd(m2)
    st["sppf.idx"] = (i1, i2, i3)
    st["sppf.cat"] = np.concatenate([s1, m1, m2, m3], axis=-1)
    st["b9.cv2.shape"], st["b9.cv2"] = _conv("b9.cv2", st["sppf.cat"], P, eps, 1)
    a9 = st["b9.cv2"]["a"]
    a6, a4 = st["b6"]["out"], st["b4"]["out"]
    st["n12.in"] = np.concatenate([upsample2x_fwd(a9), a6], axis=-1)
    st["n12"] = _c2f("n12", st["n12.in"], P, eps)
    a12 = st["n12"]["out"]
    st["n15.in"] = np.concatenate([upsample2x_fwd(a12), a4], axis=-1)
    st["n15"] = _c2f("n15", st["n15.in"], P, eps)
    a15 = st["n15"]["out"]
    st["n16.shape"], st["n16"] = _conv("n16", a15, P, eps, 2)
    st["n18.in"] = np.concatenate([st["n16"]["a"], a12], axis=-1)
    st["n18"] = _c2f("n18", st["n18.in"], P, eps)
    a18 = st["n18"]["out"]
    st["n19.shape"], st["n19"] = _conv("n19", a18, P, eps, 2)
    st["n21.in"] = np.concatenate([st["n19"]["a"], a9], axis=-1)
    st["n21"] = _c2f("n21", st["n21.in"], P, eps)
    st["P3"], st["P4"], st["P5"] = a15, a18, st["n21"]["out"]
    return st


def backward(g3, g4, g5, st, P, eps):
    """Returns (grads: layer name -> dict(dw, dgamma, dbeta, ...), dx of the image)."""
    G = {}

    def c2f_b(prefix, gout):
        nb, sc = C2F[prefix]
        names, params = _c2f_params(prefix, P)
        x = st[prefix + ".in"]
        n, h, _, c1 = x.shape
        c2 = params[-1][0].shape[0]
        grads, dx = c2f_bwd(gout, st[prefix], params, n, h, c1, c2, nb, eps, sc)
        G.update(dict(zip(names, grads)))
        return dx

    def conv_b(name, gout, x):
        w, ga, be = P[name]
        G[name] = block_bwd(gout, x, w, st[name + ".shape"], st[name], ga, be, eps)
        return G[name]["dx"]

    c9 = st["b9.cv2"]["a"].shape[-1]
    c19 = st["n19"]["a"].shape[-1]
    c16 = st["n16"]["a"].shape[-1]
    d20 = c2f_b("n21", g5)
    d9 = d20[..., c19:].copy()
    d18 = np.asarray(g4, np.float64) + conv_b("n19", d20[..., :c19], st["n18"]["out"])
    d17 = c2f_b("n18", d18)
    d12 = d17[..., c16:].copy()
    d15 = np.asarray(g3, np.float64) + conv_b("n16", d17[..., :c16], st["n15"]["out"])
    d14 = c2f_b("n15", d15)
    c13 = st["n12"]["out"].shape[-1]
    d4 = d14[..., c13:].copy()
    d12 = d12 + upsample2x_bwd(d14[..., :c13])
    d11 = c2f_b("n12", d12)
    d6 = d11[..., c9:].copy()
    d9 = d9 + upsample2x_bwd(d11[..., :c9])
    dcat = conv_b("b9.cv2", d9, st["sppf.cat"])
    q = dcat.shape[-1] // 4
    ds, dm1, dm2, dm3 = (dcat[..., k * q:(k + 1) * q].copy() for k in range(4))
    i1, i2, i3 = st["sppf.idx"]
    dm2 = dm2 + maxpool_bwd(dm3, i3)
    dm1 = dm1 + maxpool_bwd(dm2, i2)
    ds = ds + maxpool_bwd(dm1, i1)
    d8 = conv_b("b9.cv1", ds, st["b9.in"])
    d7 = c2f_b("b8", d8)
    d6 = d6 + conv_b("b7", d7, st["b7.in"])
    d5 = c2f_b("b6", d6)
    d4 = d4 + conv_b("b5", d5, st["b5.in"])
    d3 = c2f_b("b4", d4)
    d2 = conv_b("b3", d3, st["b3.in"])
    d1 = c2f_b("b2", d2)
    d0 = conv_b("b1", d1, st["b1.in"])
    dx = conv_b("b0", d0, st["b0.in"])
    return G, dx
