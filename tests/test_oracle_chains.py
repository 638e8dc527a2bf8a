"""Pins of the block and multi-block oracles (one Conv+BN+SiLU block, the stem
chain, the C2f block) against torch float64 autograd and finite differences."""
import numpy as np
import pytest
import torch

import oracle
from oracle import ConvShape, chains

EPS = 1e-3
F = torch.nn.functional


def t(a, grad=False):
    return torch.from_numpy(np.ascontiguousarray(a)).requires_grad_(grad)


def torch_block(x, w, gamma, beta, s: ConvShape, residual=None):
    """NHWC in/out, float64."""
    y = F.conv2d(x.permute(0, 3, 1, 2), w.permute(0, 3, 1, 2), stride=(s.sh, s.sw), padding=(s.ph, s.pw))
    a = F.silu(F.batch_norm(y, None, None, gamma, beta, training=True, eps=EPS)).permute(0, 2, 3, 1)
    return a + residual if residual is not None else a


def test_block_fd_and_torch():
    s = ConvShape(2, 5, 6, 3, 4, 3, 3, 2, 2, 1, 1)
    r = np.random.default_rng(0)
    x, w = r.standard_normal(s.x_shape), r.uniform(-0.3, 0.3, s.w_shape)
    gamma, beta = r.uniform(0.5, 1.5, 4), r.normal(0, 0.2, 4)
    g = r.standard_normal(s.y_shape)
    f = oracle.block_fwd(x, w, s, gamma, beta, EPS)
    b = oracle.block_bwd(g, x, w, s, f, gamma, beta, EPS)
    xt, wt, gt, bt = t(x, True), t(w, True), t(gamma, True), t(beta, True)
    at = torch_block(xt, wt, gt, bt, s)
    at.backward(t(g))
    np.testing.assert_allclose(f["a"], at.detach().numpy(), atol=1e-12)
    for mine, ref in ((b["dx"], xt.grad), (b["dw"], wt.grad), (b["dgamma"], gt.grad), (b["dbeta"], bt.grad)):
        ref = ref.numpy()
        np.testing.assert_allclose(mine, ref, atol=1e-10 * np.abs(ref).max())

    # central differences on a handful of coordinates of x and w
    def L():
        return float(np.sum(g * oracle.block_fwd(x, w, s, gamma, beta, EPS)["a"]))

    h = 1e-6
    for arr, grad in ((x, b["dx"]), (w, b["dw"])):
        for i in np.random.default_rng(1).integers(0, arr.size, 8):
            old = arr.flat[i]
            arr.flat[i] = old + h
            lp = L()
            arr.flat[i] = old - h
            lm = L()
            arr.flat[i] = old
            assert abs((lp - lm) / (2 * h) - grad.flat[i]) < 1e-6 * max(1.0, np.abs(grad).max())


def test_stem_chain_matches_torch():
    s0 = ConvShape(2, 12, 12, 3, 8, 3, 3, 2, 2, 1, 1)
    s1 = ConvShape(2, 6, 6, 8, 16, 3, 3, 2, 2, 1, 1)
    r = np.random.default_rng(2)
    x = r.uniform(0, 1, s0.x_shape)
    ws = [r.uniform(-1 / np.sqrt(27), 1 / np.sqrt(27), s0.w_shape), r.uniform(-1 / 12, 1 / 12, s1.w_shape)]
    gs, bs = [np.ones(8), np.ones(16)], [np.zeros(8), np.zeros(16)]
    acts, fwds = chains.chain_fwd(x, ws, [s0, s1], gs, bs, EPS)
    g = r.standard_normal(acts[-1].shape)
    grads, dx = chains.chain_bwd(g, acts, fwds, ws, [s0, s1], gs, bs, EPS)
    xt = t(x, True)
    wts = [t(w, True) for w in ws]
    a = torch_block(torch_block(xt, wts[0], t(gs[0]), t(bs[0]), s0), wts[1], t(gs[1]), t(bs[1]), s1)
    a.backward(t(g))
    np.testing.assert_allclose(acts[-1], a.detach().numpy(), atol=1e-12)
    np.testing.assert_allclose(dx, xt.grad.numpy(), atol=1e-10 * np.abs(dx).max())
    for gr, wt in zip(grads, wts):
        np.testing.assert_allclose(gr["dw"], wt.grad.numpy(), atol=1e-10 * np.abs(gr["dw"]).max())


@pytest.mark.parametrize("shortcut", [True, False])
def test_c2f_matches_torch(shortcut):
    n, h, c1, c2, nb = 2, 6, 8, 8, 2
    cv1, m, cv2 = chains.c2f_shapes(n, h, c1, c2, nb)
    r = np.random.default_rng(3)
    shapes = [cv1] + [m] * (2 * nb) + [cv2]
    params = [(r.uniform(-0.5, 0.5, s.w_shape), r.uniform(0.5, 1.5, s.co), r.normal(0, 0.2, s.co)) for s in shapes]
    x = r.standard_normal((n, h, h, c1))
    st = chains.c2f_fwd(x, params, n, h, c1, c2, nb, EPS, shortcut)
    g = r.standard_normal(st["out"].shape)
    grads, dx = chains.c2f_bwd(g, st, params, n, h, c1, c2, nb, EPS, shortcut)

    xt = t(x, True)
    tp = [(t(w, True), t(ga, True), t(be, True)) for w, ga, be in params]
    a = torch_block(xt, *tp[0], cv1)
    pieces = [a[..., :c2 // 2], a[..., c2 // 2:]]
    for i in range(nb):
        inp = pieces[-1]
        u = torch_block(inp, *tp[1 + 2 * i], m)
        pieces.append(torch_block(u, *tp[2 + 2 * i], m, residual=inp if shortcut else None))
    out = torch_block(torch.cat(pieces, -1), *tp[-1], cv2)
    out.backward(t(g))
    np.testing.assert_allclose(st["out"], out.detach().numpy(), atol=1e-12)
    np.testing.assert_allclose(dx, xt.grad.numpy(), atol=1e-10 * np.abs(dx).max())
    for gr, (wt, gt, bt) in zip(grads, tp):
        np.testing.assert_allclose(gr["dw"], wt.grad.numpy(), atol=1e-10 * np.abs(gr["dw"]).max())
        np.testing.assert_allclose(gr["dgamma"], gt.grad.numpy(), atol=1e-10 * np.abs(gr["dgamma"]).max())
        np.testing.assert_allclose(gr["dbeta"], bt.grad.numpy(), atol=1e-10 * np.abs(gr["dbeta"]).max())
