"""GPU parity of prologue fusion in the 3x3 stride-1 halo kernel.

Forward (the previous layer's BN + SiLU applied inside the convolution's operand staging):
against the fp64 oracle's composition conv(SiLU(BN(y_prev))) element by element (rel_inf
<= 2e-2 on y, and on the batch statistics: the fused activations are rounded to bf16 before
the convolution, as the unfused path's stored activations are, while the oracle's are
exact), and bit for bit against numbat_bn_silu_fwd followed by numbat_conv_fwd where that
forward runs the same kernel (grids of at least 256 tiles).

Backward (the layer's BN + SiLU backward formed inside the data gradient's operand staging,
dy written out as well): dy against the oracle's BN + SiLU backward and dx against the
oracle's data gradient of that dy (stage-isolated: the oracle takes the GPU's bf16 dy),
element by element at rel_inf <= 2e-2, every pixel of dy written and the channels past
c_out of strided tensors untouched; and dx and dy bit for bit against numbat_bn_silu_bwd
followed by numbat_conv_bwd_data at the detector's full layer sizes."""
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


# ---- backward: dy = BN+SiLU backward(g, y) formed in the data gradient's halo staging

def make_bwd(case, idx):
    n, h, w, ci, co, gs, ys, acc = case
    inp = Inputs(121, idx)
    yb = inp.normal((n, h, w, co), synth.T_Y, -0.1, 1.4)
    gb = inp.normal((n, h, w, co), synth.T_G)
    wb = inp.weight(co, 3, ci)
    gamma = inp.f32_uniform((co,), synth.T_GAMMA, 0.5, 1.5)
    beta = inp.f32_normal((co,), synth.T_BETA, 0.0, 0.3)
    dx0 = inp.normal((n, h, w, ci), synth.T_RES)
    return yb, gb, wb, gamma, beta, dx0


def strided(bits, stride, fill=0x7fc0):
    """bf16 bits [..., c] placed in the first c channels of a [..., stride] device tensor
    (the rest holds `fill`, a NaN by default)"""
    if stride == 0 or stride == bits.shape[-1]:
        return blocks.dev_bf16(bits)
    full = np.full(bits.shape[:-1] + (stride,), fill, np.uint16)
    full[..., :bits.shape[-1]] = bits
    return blocks.dev_bf16(full)


def bn_state(n, h, w, co, ys, gs, y, gamma, beta):
    """save_mean / save_rstd from the BN forward, then dgamma / dbeta from the BN backward
    without dy (what the fused data gradient takes)"""
    bnp = nb.bn_problem(n * h * w, co, eps=EPS, y_pixel_stride=ys, a_pixel_stride=gs, dy_pixel_stride=ys)
    ws = blocks.workspace(max(nb.numbat_workspace_size(nb.OP_BN_SILU_FWD, bnp),
                              nb.numbat_workspace_size(nb.OP_BN_SILU_BWD, bnp)))
    out = torch.empty((n, h, w, ys or co), dtype=torch.bfloat16, device="cuda")
    sm, sr = torch.empty(co, device="cuda"), torch.empty(co, device="cuda")
    nb.numbat_bn_silu_fwd(nb.bn_problem(n * h * w, co, eps=EPS, y_pixel_stride=ys, a_pixel_stride=ys), y, None,
                          gamma, beta, None, out, sm, sr, ws=ws)
    return bnp, ws, sm, sr


# n, h, w, c_in, c_out, g pixel stride, y / dy pixel stride, accumulate into dx: every halo
# tile shape (128 x 96 and 128 x 64 linear tiles up to 63 wide, 256-row ones up to 95,
# 8 x 32 tiles of wider images, with 96 and 64 columns), chunk tails (48 and 80 channels),
# ragged last tiles, strided g and y, accumulation
BWD_CASES = [
    (2, 20, 20, 96, 288, 0, 0, False),
    (3, 13, 11, 64, 48, 0, 0, False),
    (1, 40, 40, 192, 192, 0, 0, True),
    (2, 30, 80, 96, 96, 0, 0, False),
    (2, 17, 70, 64, 64, 0, 0, False),
    (1, 16, 160, 48, 48, 0, 0, False),
    (1, 8, 128, 96, 96, 0, 0, True),
    (2, 21, 19, 96, 80, 112, 96, False),
    (2, 16, 96, 64, 32, 64, 48, True),
]


@pytest.mark.parametrize("i", range(len(BWD_CASES)),
                         ids=["n{}h{}w{}ci{}co{}gs{}ys{}acc{:d}".format(*c) for c in BWD_CASES])
def test_prologue_backward_matches_oracle(i):
    case = BWD_CASES[i]
    n, h, w, ci, co, gs, ys, acc = case
    yb, gb, wb, gamma, beta, dx0 = make_bwd(case, i)
    y, g = strided(yb, ys), strided(gb, gs)
    ga, be = blocks.dev_f32(gamma), blocks.dev_f32(beta)
    bnp, ws, sm, sr = bn_state(n, h, w, co, ys, gs, y, ga, be)
    dg, db = torch.empty(co, device="cuda"), torch.empty(co, device="cuda")
    nb.numbat_bn_silu_bwd(bnp, g, y, sm, sr, ga, be, None, dg, db, None, ws=ws)
    prob = nb.conv_problem(n, h, w, ci, co, 3, y_pixel_stride=ys)
    assert nb.numbat_workspace_size(nb.OP_CONV_BWD_DATA_BN_SILU, prob) == 0
    dy = torch.full((n, h, w, ys or co), float("nan"), dtype=torch.bfloat16, device="cuda")
    dx = blocks.dev_bf16(dx0) if acc else torch.full((n, h, w, ci), float("nan"), dtype=torch.bfloat16,
                                                     device="cuda")
    print(f"prologue backward {case}: launching", flush=True)
    nb.numbat_conv_bwd_data_bn_silu_prologue(prob, g, y, sm, sr, ga, be, dg, db, blocks.dev_bf16(wb), dx, dy,
                                             accumulate=acc, g_pixel_stride=gs)
    torch.cuda.synchronize()
    dyh = blocks.host_f64(dy)
    mref, vref = oracle.bn_stats(f64(yb))
    dyr, dgr, dbr = oracle.bn_silu_bwd(f64(gb), f64(yb), mref, vref, gamma.astype(np.float64),
                                       beta.astype(np.float64), EPS)
    ed = assert_close(dyh[..., :co], dyr, "dy")
    if ys and ys > co:
        assert np.isnan(dyh[..., co:]).all(), "dy channels past c_out were written"
    s = ConvShape(n, h, w, ci, co, 3, 3, 1, 1, 1, 1)
    dxr = oracle.conv_dgrad(dyh[..., :co], f64(wb), s)
    if acc:
        dxr = dxr + f64(dx0)
    ex = assert_close(blocks.host_f64(dx), dxr, "dx")
    print(f"prologue backward {case}: dy rel_inf {ed:.1e}, dx rel_inf {ex:.1e}", flush=True)


# the detector's 3x3 stride-1 layer sizes at batch 16 (160 x 160 x 48, 80 x 80 x 96,
# 40 x 40 x 192, 20 x 20 x 288, and a head layer's 40 x 40 x 64)
BWD_BITWISE = [(16, 160, 160, 48, 48), (16, 80, 80, 96, 96), (16, 40, 40, 192, 192), (16, 20, 20, 288, 288),
               (16, 40, 40, 64, 64)]


@pytest.mark.parametrize("i", range(len(BWD_BITWISE)), ids=["n{}h{}w{}ci{}co{}".format(*c) for c in BWD_BITWISE])
def test_prologue_backward_equals_bn_then_dgrad_bitwise(i):
    n, h, w, ci, co = BWD_BITWISE[i]
    yb, gb, wb, gamma, beta, _ = make_bwd((n, h, w, ci, co, 0, 0, False), 20 + i)
    y, g, wt = blocks.dev_bf16(yb), blocks.dev_bf16(gb), blocks.dev_bf16(wb)
    ga, be = blocks.dev_f32(gamma), blocks.dev_f32(beta)
    bnp, ws, sm, sr = bn_state(n, h, w, co, 0, 0, y, ga, be)
    prob = nb.conv_problem(n, h, w, ci, co, 3)
    # unfused: BN + SiLU backward (writes dy), then the data gradient
    dy1 = torch.full((n, h, w, co), float("nan"), dtype=torch.bfloat16, device="cuda")
    dg1, db1 = torch.empty(co, device="cuda"), torch.empty(co, device="cuda")
    nb.numbat_bn_silu_bwd(bnp, g, y, sm, sr, ga, be, dy1, dg1, db1, None, ws=ws)
    dx1 = torch.full((n, h, w, ci), float("nan"), dtype=torch.bfloat16, device="cuda")
    wsd = blocks.workspace(nb.numbat_workspace_size(nb.OP_CONV_BWD_DATA, prob))
    nb.numbat_conv_bwd_data(prob, dy1, wt, dx1, False, wsd)
    # fused
    dg2, db2 = torch.empty(co, device="cuda"), torch.empty(co, device="cuda")
    nb.numbat_bn_silu_bwd(bnp, g, y, sm, sr, ga, be, None, dg2, db2, None, ws=ws)
    dy2, dx2 = torch.full_like(dy1, float("nan")), torch.full_like(dx1, float("nan"))
    nb.numbat_conv_bwd_data_bn_silu_prologue(prob, g, y, sm, sr, ga, be, dg2, db2, wt, dx2, dy2)
    torch.cuda.synchronize()
    print(f"prologue backward bitwise {BWD_BITWISE[i]}: dgamma/dbeta equal {torch.equal(dg1, dg2)}/"
          f"{torch.equal(db1, db2)}, dy equal {torch.equal(dy1, dy2)}, dx equal {torch.equal(dx1, dx2)}", flush=True)
    assert torch.equal(dg1, dg2) and torch.equal(db1, db2)
    assert torch.equal(dy1, dy2), rel_inf(blocks.host_f64(dy2), blocks.host_f64(dy1))
    assert torch.equal(dx1, dx2), rel_inf(blocks.host_f64(dx2), blocks.host_f64(dx1))
