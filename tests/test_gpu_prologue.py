"""GPU parity of the prologue-fused forward (the previous layer's BN + SiLU applied inside the
3x3 stride-1 convolution's operand staging): against the fp64 oracle's composition
conv(SiLU(BN(y_prev))) element by element (rel_inf <= 2e-2 on y, and on the batch
statistics: the fused activations are rounded to bf16 before the convolution, as the
unfused path's stored activations are, while the oracle's are exact), and bit for bit
against numbat_bn_silu_fwd followed by numbat_conv_fwd where that forward runs the same
kernel (grids of at least 256 tiles)."""
import numpy as np
import pytest

import oracle
from oracle import ConvShape
from parity import Inputs, assert_close, f64, rel_inf
from paper_2609_10632_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    from paper_2609_10632_amd import blocks
    from paper_2609_10632_amd import numbat as nb

EPS = 1e-3


def make(case, idx):
    n, h, w, ci, co = case
    inp = Inputs(120, idx)
    yb = inp.normal((n, h, w, ci), synth.T_Y, 0.1, 1.3)
    wb = inp.weight(co, 3, ci)
    mean = inp.f32_normal((ci,), synth.T_MEAN, 0.1, 0.2)
    var = inp.f32_uniform((ci,), synth.T_VAR, 0.5, 2.0)
    gamma = inp.f32_uniform((ci,), synth.T_GAMMA, 0.5, 1.5)
    beta = inp.f32_normal((ci,), synth.T_BETA, 0.0, 0.1)
    return yb, wb, mean, var, gamma, beta


def run_fused(case, yb, wb, mean, var, gamma, beta):
    n, h, w, ci, co = case
    blk = blocks.ConvBlock(n, h, w, ci, co, 3, 1)
    y = torch.full((n, h, w, co), float("nan"), dtype=torch.bfloat16, device="cuda")
    st = torch.full((2 * co,), float("nan"), device="cuda")
    prev = torch.from_numpy(np.concatenate([mean, var]).astype(np.float32)).cuda()
    nb.numbat_conv_fwd_bn_silu_prologue(blk.prob, blocks.dev_bf16(yb), prev, torch.from_numpy(gamma).cuda(),
                                        torch.from_numpy(beta).cuda(), EPS, blocks.dev_bf16(wb), y, st,
                                        blocks.workspace(blk.ws_fwd))
    return blk, y, st


# n, h, w, c_in, c_out: linear tiles on 128 and 256 rows, small grids (the halo kernel on any
# grid), chunk tails (48, 80 channels), several images per tile, 2D 8 x 32 tiles
CASES = [
    (2, 20, 20, 288, 96),
    (3, 5, 3, 32, 64),
    (2, 21, 19, 80, 48),
    (1, 40, 40, 192, 192),
    (2, 30, 80, 96, 96),
    (3, 16, 96, 48, 64),
    (1, 64, 128, 48, 96),
]


@pytest.mark.parametrize("i", range(len(CASES)), ids=["n{}h{}w{}ci{}co{}".format(*c) for c in CASES])
def test_prologue_forward_matches_oracle(i):
    case = CASES[i]
    n, h, w, ci, co = case
    yb, wb, mean, var, gamma, beta = make(case, i)
    blk, y, st = run_fused(case, yb, wb, mean, var, gamma, beta)
    torch.cuda.synchronize()
    a = oracle.bn_silu_fwd(f64(yb), mean.astype(np.float64), var.astype(np.float64), gamma.astype(np.float64),
                           beta.astype(np.float64), EPS)
    s = ConvShape(n, h, w, ci, co, 3, 3, 1, 1, 1, 1)
    yref = oracle.conv_fwd(a, f64(wb), s)
    e = assert_close(blocks.host_f64(y), yref, "y")
    mref, vref = oracle.bn_stats(yref)
    stg = blocks.host_f64(st)
    em = np.abs(stg[:co] - mref).max() / np.sqrt(vref + EPS).max()
    ev = np.abs(stg[co:] - vref).max() / vref.max()
    assert em <= 2e-2 and ev <= 2e-2, (em, ev)
    print(f"prologue {case}: y rel_inf {e:.1e}, stats mean {em:.1e} var {ev:.1e}", flush=True)


# grids of at least 256 tiles, where numbat_conv_fwd runs the same halo kernel
BITWISE = [(8, 66, 63, 32, 96), (16, 40, 40, 192, 192), (4, 160, 160, 48, 48)]


@pytest.mark.parametrize("i", range(len(BITWISE)), ids=["n{}h{}w{}ci{}co{}".format(*c) for c in BITWISE])
def test_prologue_forward_equals_bn_then_conv_bitwise(i):
    case = BITWISE[i]
    n, h, w, ci, co = case
    yb, wb, mean, var, gamma, beta = make(case, 10 + i)
    blk, y2, st2 = run_fused(case, yb, wb, mean, var, gamma, beta)
    # unfused: BN + SiLU of the previous layer (writes the activation), then the forward
    bnp = nb.bn_problem(n * h * w, ci, eps=EPS)
    prev = torch.from_numpy(np.concatenate([mean, var]).astype(np.float32)).cuda()
    act = torch.empty((n, h, w, ci), dtype=torch.bfloat16, device="cuda")
    sm, sr = torch.empty(ci, device="cuda"), torch.empty(ci, device="cuda")
    nb.numbat_bn_silu_fwd(bnp, blocks.dev_bf16(yb), prev, torch.from_numpy(gamma).cuda(),
                          torch.from_numpy(beta).cuda(), None, act, sm, sr)
    y1 = torch.full_like(y2, float("nan"))
    st1 = torch.full_like(st2, float("nan"))
    nb.numbat_conv_fwd(blk.prob, act, blocks.dev_bf16(wb), y1, st1, blocks.workspace(blk.ws_fwd))
    torch.cuda.synchronize()
    print(f"prologue bitwise {case}: y equal {torch.equal(y1, y2)}, stats equal {torch.equal(st1, st2)}", flush=True)
    assert torch.equal(y1, y2), rel_inf(blocks.host_f64(y2), blocks.host_f64(y1))
    assert torch.equal(st1, st2)
