"""Pins of the inference-mode oracle pieces: conv with bias and eval-mode BN+SiLU against
torch's conv2d (bias) and batch_norm(training=False) + silu in float64, the eval formula
reducing to the identity's SiLU when the running statistics are (0, 1 - eps) and gamma/beta
are (1, 0), and the head composition against torch layers built from the same parameters."""
import numpy as np
import pytest

import oracle
from oracle import ConvShape, head

torch = pytest.importorskip("torch")
F = torch.nn.functional


def t64(a):
    return torch.tensor(np.asarray(a), dtype=torch.float64)


def nchw(a):
    return t64(a).permute(0, 3, 1, 2)


def test_conv_bias_matches_torch():
    rng = np.random.default_rng(0)
    x, w, b = rng.standard_normal((2, 7, 9, 16)), rng.standard_normal((24, 1, 1, 16)), rng.standard_normal(24)
    s = ConvShape(2, 7, 9, 16, 24, 1, 1)
    ref = F.conv2d(nchw(x), t64(w).permute(0, 3, 1, 2), t64(b)).permute(0, 2, 3, 1).numpy()
    assert np.allclose(oracle.conv_fwd_bias(x, w, b, s), ref, rtol=1e-13, atol=1e-13)


def test_bn_silu_eval_matches_torch_and_closed_form():
    rng = np.random.default_rng(1)
    y = rng.standard_normal((300, 40)) * 2 + 0.5
    rm, rv = rng.standard_normal(40) * 0.3, rng.uniform(0.2, 3.0, 40)
    g, b = rng.uniform(0.5, 1.5, 40), rng.standard_normal(40) * 0.1
    ref = F.silu(F.batch_norm(t64(y), t64(rm), t64(rv), t64(g), t64(b), training=False, eps=1e-3)).numpy()
    assert np.allclose(oracle.bn_silu_eval(y, rm, rv, g, b, 1e-3), ref, rtol=1e-13, atol=1e-13)
    # running statistics (0, 1 - eps), gamma 1, beta 0: a = SiLU(y) exactly
    a = oracle.bn_silu_eval(y, np.zeros(40), np.full(40, 1 - 1e-3), np.ones(40), np.zeros(40), 1e-3)
    assert np.allclose(a, y / (1 + np.exp(-y)), rtol=1e-15, atol=1e-15)
    # training mode is different: eval uses the running, not the batch, statistics
    mean, var = oracle.bn_stats(y)
    assert np.abs(oracle.bn_silu_fwd(y, mean, var, g, b, 1e-3) - oracle.bn_silu_eval(y, rm, rv, g, b, 1e-3)).max() > 0.1


def test_head_matches_torch_layers():
    rng = np.random.default_rng(2)
    c, eps = 32, 1e-3

    def conv_bn(ci, co, k):
        return {"w": rng.standard_normal((co, k, k, ci)) * 0.2, "gamma": rng.uniform(0.5, 1.5, co),
                "beta": rng.standard_normal(co) * 0.1, "mean": rng.standard_normal(co) * 0.1,
                "var": rng.uniform(0.5, 2.0, co)}

    box = [conv_bn(c, 64, 3), conv_bn(64, 64, 3), {"w": rng.standard_normal((64, 1, 1, 64)) * 0.1,
                                                  "bias": rng.standard_normal(64)}]
    cls = [conv_bn(c, 192, 3), conv_bn(192, 192, 3), {"w": rng.standard_normal((80, 1, 1, 192)) * 0.1,
                                                      "bias": rng.standard_normal(80)}]
    x = rng.standard_normal((1, 6, 5, c))

    def torch_branch(a, layers):
        for L in layers:
            w = t64(L["w"]).permute(0, 3, 1, 2)
            if "bias" in L:
                a = F.conv2d(a, w, t64(L["bias"]))
            else:
                a = F.silu(F.batch_norm(F.conv2d(a, w, padding=w.shape[-1] // 2), t64(L["mean"]), t64(L["var"]),
                                        t64(L["gamma"]), t64(L["beta"]), training=False, eps=eps))
        return a

    ref = torch.cat([torch_branch(nchw(x), box), torch_branch(nchw(x), cls)], 1).permute(0, 2, 3, 1).numpy()
    got = head.head_infer(x, box, cls, eps)
    assert got.shape == (1, 6, 5, 144)
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)
