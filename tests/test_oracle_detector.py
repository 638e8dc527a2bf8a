"""Pin of the chain-mode detector oracle (backbone + neck dataflow) against torch autograd
of the same network written with torch's own ops (conv2d, batch_norm in training mode, silu,
max_pool2d, nearest interpolate, cat) in float64, at batch 1 and a 64x64 input: the three
outputs, the image gradient and every layer's dw, dgamma and dbeta."""
import numpy as np
import pytest

from oracle import detector
from paper_2609_10632_amd import workloads

torch = pytest.importorskip("torch")
F = torch.nn.functional
EPS = 1e-3


def params(seed):
    rng = np.random.default_rng(seed)
    P = {}
    for l in workloads.backbone_neck_layers():
        b = 1.0 / np.sqrt(l.ci * l.k * l.k)
        P[l.name] = (rng.uniform(-b, b, (l.co, l.k, l.k, l.ci)), rng.uniform(0.5, 1.5, l.co),
                     rng.normal(0, 0.1, l.co))
    return P


def torch_net(x, T):
    def cbs(a, name, stride=1, res=None):
        w, g, b = T[name]
        y = F.conv2d(a, w, stride=stride, padding=w.shape[-1] // 2)
        o = F.silu(F.batch_norm(y, None, None, g, b, training=True, eps=EPS))
        return o + res if res is not None else o

    def c2f(a, prefix):
        nb, sc = detector.C2F[prefix]
        t = cbs(a, f"{prefix}.cv1")
        half = t.shape[1] // 2
        pieces = [t[:, :half], t[:, half:]]
        for i in range(nb):
            inp = pieces[-1]
            u = cbs(inp, f"{prefix}.m{i}.cv1")
            pieces.append(cbs(u, f"{prefix}.m{i}.cv2", res=inp if sc else None))
        return cbs(torch.cat(pieces, 1), f"{prefix}.cv2")

    up = lambda a: F.interpolate(a, scale_factor=2, mode="nearest")
    pool = lambda a: F.max_pool2d(a, 5, 1, 2)
    a = cbs(cbs(x, "b0", 2), "b1", 2)
    a4 = c2f(cbs(c2f(a, "b2"), "b3", 2), "b4")
    a6 = c2f(cbs(a4, "b5", 2), "b6")
    a8 = c2f(cbs(a6, "b7", 2), "b8")
    s = cbs(a8, "b9.cv1")
    m1 = pool(s)
    m2 = pool(m1)
    a9 = cbs(torch.cat([s, m1, m2, pool(m2)], 1), "b9.cv2")
    a12 = c2f(torch.cat([up(a9), a6], 1), "n12")
    a15 = c2f(torch.cat([up(a12), a4], 1), "n15")
    a18 = c2f(torch.cat([cbs(a15, "n16", 2), a12], 1), "n18")
    a21 = c2f(torch.cat([cbs(a18, "n19", 2), a9], 1), "n21")
    return a15, a18, a21


def test_detector_matches_torch_autograd():
    P = params(0)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((1, 64, 64, 3))
    st = detector.forward(x, P, EPS)
    gs = [rng.standard_normal(st[k].shape) for k in ("P3", "P4", "P5")]
    G, dx = detector.backward(*gs, st, P, EPS)

    T = {k: tuple(torch.tensor(v if i else v.transpose(0, 3, 1, 2), dtype=torch.float64, requires_grad=True)
                  for i, v in enumerate(p)) for k, p in P.items()}
    xt = torch.tensor(x.transpose(0, 3, 1, 2), dtype=torch.float64, requires_grad=True)
    outs = torch_net(xt, T)
    loss = sum((o * torch.tensor(g.transpose(0, 3, 1, 2))).sum() for o, g in zip(outs, gs))
    loss.backward()
    # relative to the largest magnitude of each quantity (the two sides sum in different orders)
    rel = lambda a, b: float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-30))
    for o, k in zip(outs, ("P3", "P4", "P5")):
        assert rel(st[k], o.detach().numpy().transpose(0, 2, 3, 1)) <= 1e-9, k
    assert rel(dx, xt.grad.numpy().transpose(0, 2, 3, 1)) <= 1e-9
    for name, (tw, tg, tb) in T.items():
        assert rel(G[name]["dw"], tw.grad.numpy().transpose(0, 2, 3, 1)) <= 1e-9, name
        assert rel(G[name]["dgamma"], tg.grad.numpy()) <= 1e-9, name
        assert rel(G[name]["dbeta"], tb.grad.numpy()) <= 1e-9, name
