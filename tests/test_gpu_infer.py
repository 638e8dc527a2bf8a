"""GPU parity of the inference-mode path against the fp64 oracle: conv with bias, Conv+BN+SiLU
with running statistics folded into the conv output stage, standalone eval BN+SiLU (with
residual and channel views), and the faithful decoupled detect head at its three scales.
Tolerance: rel_inf <= 2e-2 on every bf16 output."""
import numpy as np
import pytest

import oracle
from oracle import ConvShape, head
from parity import Inputs, assert_close, f64, report
from paper_2609_10632_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    from paper_2609_10632_amd import blocks
    from paper_2609_10632_amd import numbat as nb

EPS = 1e-3
# n, h, ci, co, k, s: 1x1 prediction convs, 3x3 (halo and direct-to-LDS), stride 2, the image layer
CASES = [(2, 20, 64, 64, 1, 1), (2, 20, 192, 80, 1, 1), (2, 40, 192, 96, 3, 1), (4, 66, 32, 96, 3, 1),
         (2, 21, 48, 64, 3, 2), (2, 32, 3, 48, 3, 2), (1, 13, 96, 40, 3, 1)]


def bn_params(ip, co):
    return (ip.f32_uniform((co,), synth.T_GAMMA, 0.5, 1.5), ip.f32_normal((co,), synth.T_BETA, 0.0, 0.1),
            ip.f32_normal((co,), synth.T_MEAN, 0.0, 0.2), ip.f32_uniform((co,), synth.T_VAR, 0.3, 2.0))


@pytest.mark.parametrize("i", range(len(CASES)), ids=["n{}h{}ci{}co{}k{}s{}".format(*c) for c in CASES])
def test_conv_bias_and_conv_bn_silu_infer(i):
    n, h, ci, co, k, st = CASES[i]
    s = ConvShape(n, h, h, ci, co, k, k, st, st, k // 2, k // 2)
    ip = Inputs(120, i)
    xb, wb = ip.normal(s.x_shape, synth.T_X), ip.weight(co, k, ci)
    bias = ip.f32_normal((co,), synth.T_BETA, 0.0, 0.5)
    g, b, m, v = bn_params(ip, co)
    p = nb.conv_problem(n, h, h, ci, co, k, stride=st)
    x, w = blocks.dev_bf16(xb), blocks.dev_bf16(wb)
    y1 = torch.empty(s.y_shape, dtype=torch.bfloat16, device="cuda")
    y2 = torch.empty_like(y1)
    nb.numbat_conv_fwd_bias(p, x, w, blocks.dev_f32(bias), y1)
    nb.numbat_conv_bn_silu_infer(p, x, w, blocks.dev_f32(g), blocks.dev_f32(b), blocks.dev_f32(m), blocks.dev_f32(v),
                                 EPS, y2)
    torch.cuda.synchronize()
    yref = oracle.conv_fwd(f64(xb), f64(wb), s)
    e1 = assert_close(blocks.host_f64(y1), yref + bias.astype(np.float64), "conv + bias")
    aref = oracle.bn_silu_eval(yref, m.astype(np.float64), v.astype(np.float64), g.astype(np.float64),
                               b.astype(np.float64), EPS)
    e2 = assert_close(blocks.host_f64(y2), aref, "conv + eval BN + SiLU")
    report(f"infer {CASES[i]} complete: conv+bias rel_inf {e1:.1e}, conv+evalBN+SiLU rel_inf {e2:.1e}")


def test_bn_silu_infer_residual_views():
    m_, c = 3000, 96
    ip = Inputs(121)
    ybig = ip.normal((m_, 192), synth.T_Y, 0.2, 1.5)
    rb = ip.normal((m_, 96), synth.T_RES)
    g, b, mu, var = bn_params(ip, c)
    p = nb.bn_problem(m_, c, EPS, y_pixel_stride=192, a_pixel_stride=288, r_pixel_stride=96)
    outbig = torch.zeros((m_, 288), dtype=torch.bfloat16, device="cuda")
    nb.numbat_bn_silu_infer(p, blocks.dev_bf16(ybig)[:, 96:], blocks.dev_f32(mu), blocks.dev_f32(var),
                            blocks.dev_f32(g), blocks.dev_f32(b), blocks.dev_bf16(rb), outbig[:, 192:])
    torch.cuda.synchronize()
    ref = oracle.bn_silu_eval(f64(ybig[:, 96:]), mu.astype(np.float64), var.astype(np.float64), g.astype(np.float64),
                              b.astype(np.float64), EPS, f64(rb))
    got = blocks.host_f64(outbig)
    assert_close(got[:, 192:], ref, "eval BN + SiLU + residual into a view")
    assert np.all(got[:, :192] == 0)


@pytest.mark.parametrize("scale", [0, 1, 2], ids=["p3_80", "p4_40", "p5_20"])
def test_faithful_head_inference(scale):
    from paper_2609_10632_amd.workloads import HEAD_SCALES

    h, c = HEAD_SCALES[scale]
    n = 2
    ip = Inputs(122, scale)
    xb = ip.normal((n, h, h, c), synth.T_X)

    def layers(widths, pred, base):
        L, ci = [], c
        for j, co in enumerate(widths):
            q = Inputs(122, 10 * scale + base + j)
            L.append((q.weight(co, 3, ci),) + bn_params(q, co))
            ci = co
        q = Inputs(122, 10 * scale + base + 5)
        L.append((q.weight(pred, 1, ci), q.f32_normal((pred,), synth.T_BETA, 0.0, 0.5)))
        return L

    box, cls = layers((64, 64), 64, 0), layers((192, 192), 80, 2)
    hd = blocks.DetectHeadInfer(n, h, c, EPS)
    dev = lambda L: [tuple(blocks.dev_bf16(t) if t.dtype == np.uint16 else blocks.dev_f32(t) for t in e) for e in L]
    out = hd.forward(blocks.dev_bf16(xb), dev(box), dev(cls))
    torch.cuda.synchronize()
    as_o = lambda L: [{"w": f64(e[0]), "gamma": e[1].astype(np.float64), "beta": e[2].astype(np.float64),
                       "mean": e[3].astype(np.float64), "var": e[4].astype(np.float64)} for e in L[:2]] + \
        [{"w": f64(L[2][0]), "bias": L[2][1].astype(np.float64)}]
    ref = head.head_infer(f64(xb), as_o(box), as_o(cls), EPS)
    eb = assert_close(blocks.host_f64(out)[..., :64], ref[..., :64], "head box output")
    ec = assert_close(blocks.host_f64(out)[..., 64:], ref[..., 64:], "head class output")
    report(f"faithful head scale {h}x{h} c={c} n={n} complete: box rel_inf {eb:.1e}, class rel_inf {ec:.1e}")
