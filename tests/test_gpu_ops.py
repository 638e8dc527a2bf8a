"""GPU parity of each C-ABI entry point against the fp64 oracle, element by element,
on seeded inputs at sizes that span several tiles and ragged tails."""
import numpy as np
import pytest

import oracle
from oracle import ConvShape
from parity import Inputs, assert_close, assert_stats, f64
from paper_2609_10632_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    from paper_2609_10632_amd import blocks
    from paper_2609_10632_amd import numbat as nb

EPS = 1e-3

# n, h, w, ci, co, k, s
CONV_CASES = [
    (2, 32, 32, 16, 32, 3, 1),
    (2, 17, 23, 3, 48, 3, 2),
    (2, 19, 21, 48, 96, 3, 2),
    (3, 13, 11, 96, 96, 1, 1),
    (2, 9, 10, 192, 80, 3, 1),
    (1, 7, 9, 64, 136, 3, 1),
    (2, 5, 5, 8, 8, 3, 1),
    (4, 20, 20, 288, 288, 3, 1),
    (1, 11, 13, 40, 24, 3, 2),
    (2, 15, 15, 3, 16, 3, 2),
    (1, 6, 6, 16, 16, 1, 2),
    (2, 12, 12, 1152, 64, 1, 1),
    # more than 32768 GEMM rows with short reductions: the direct-to-LDS kernel's
    # three-stage 32-element variant (48 channels: two tap wraps per step; 32 -> 64 stride 2:
    # 32-column data-gradient tiles)
    (2, 130, 129, 48, 48, 3, 1),
    (1, 364, 362, 32, 64, 3, 2),
    # narrow inputs (fewer than 8 channels: the image-input kernels) across channel
    # counts, kernel sizes and strides
    (2, 11, 13, 1, 8, 3, 1),
    (1, 14, 9, 5, 24, 5, 2),
    (2, 10, 10, 7, 16, 1, 1),
    (1, 13, 17, 2, 32, 3, 3),
    (1, 12, 12, 6, 40, 5, 4),
    (3, 66, 70, 3, 48, 3, 2),
    # narrow data gradients on MFMA: several patches with halos, ragged edges
    (1, 37, 75, 3, 64, 3, 1),
    (1, 41, 67, 2, 32, 3, 2),
    (1, 20, 30, 1, 16, 5, 1),
    # the image layer's forward kernel: 4 x 64 output patches
    (2, 24, 256, 3, 48, 3, 2),
    (1, 8, 128, 3, 32, 3, 2),
    # mid-size data gradient on eight-wave 256-row tiles (transposed weights), and a long
    # reduction into 384 channels on one 128 x 96 block per CU
    (2, 64, 80, 128, 128, 3, 1),
    (2, 20, 20, 384, 384, 3, 1),
    # in-place weights with an input channel count that ends mid-chunk (40 = 5 x 8), both
    # strides
    (2, 14, 10, 40, 48, 3, 1),
    (2, 15, 17, 40, 32, 3, 2),
    # c_out of 192 and 576 (three and nine 64-channel weight-gradient tiles): 3x3, a ragged
    # 1800-column reduction at stride 2, and 1x1
    (2, 10, 12, 64, 192, 3, 1),
    (1, 9, 11, 200, 576, 3, 2),
    (2, 9, 7, 576, 192, 1, 1),
    # 3x3 stride-1 halo kernel.  Data gradients always take it (up to 95-wide images);
    # forwards from 256 tiles up.  The detector's 80/40-wide shapes, tiny images (a tile
    # spans many images), chunk tails (48, 80), the widest image each tile height takes
    # (63 on 128 rows, 95 on 256) with forward grids over 256 tiles, 64-column tiles on
    # both heights; the 160- and 191-wide cases stay on the direct-to-LDS kernel
    (1, 160, 160, 48, 48, 3, 1),
    (1, 80, 80, 96, 96, 3, 1),
    (2, 40, 40, 192, 192, 3, 1),
    (3, 5, 3, 32, 64, 3, 1),
    (1, 23, 191, 64, 32, 3, 1),
    (2, 21, 19, 80, 48, 3, 1),
    (8, 66, 63, 32, 96, 3, 1),
    (6, 120, 95, 48, 96, 3, 1),
    (9, 90, 90, 32, 64, 3, 1),
    (10, 64, 60, 32, 64, 3, 1),
    # long reductions on small grids with ragged row and column tiles: 36 and 39 steps of
    # 64 (the reduction ends mid-step), stride 1 and 2
    (2, 20, 20, 256, 96, 3, 1),
    (1, 21, 19, 272, 80, 3, 1),
    (2, 41, 41, 256, 64, 3, 2),
    # two-dimensional 8 x 32 halo tiles (images wider than 95 whose width 32 divides and
    # height 8 divides): a non-square image, several small images with a 48-channel chunk
    # tail (a data gradient only: the forward grid is under 256 tiles), and a height 8 does
    # not divide (the direct-to-LDS kernel)
    (1, 64, 128, 48, 96, 3, 1),
    (3, 16, 96, 48, 64, 3, 1),
    (1, 30, 128, 32, 64, 3, 1),
    # weight gradients on 96-row output-channel tiles (four waves along k): 96 and 192
    # output channels over enough pixels that the split grid fills the GPU
    (2, 160, 160, 96, 96, 3, 1),
    (2, 160, 160, 64, 192, 3, 1),
    # patch-staged 3x3 stride-1 weight gradient (the cases above whose sides take 8 x 16,
    # 20 x 8 or 20 x 4 patches run it too): 72 of 96 output rows on 20 x 8 patches, a
    # 48-channel chunk with 40 of 64 rows on 20 x 4, one patch (a single split writes dW
    # and accumulates in place), three 48-channel chunks of a 144-channel input
    (3, 20, 24, 64, 72, 3, 1),
    (2, 40, 12, 48, 40, 3, 1),
    (1, 8, 16, 96, 32, 3, 1),
    (4, 20, 8, 144, 64, 3, 1),
    # its 1x1 form (steps of 64 pixels; the 13 x 11 and 9 x 7 cases above too): 144- and
    # 192-channel chunks (input rows padded in LDS), five 192-channel chunks into four
    # 96-row tiles, 100 steps split over many blocks, a ragged last step
    (2, 16, 16, 144, 96, 1, 1),
    (1, 20, 20, 384, 192, 1, 1),
    (1, 10, 10, 960, 384, 1, 1),
    (4, 40, 40, 288, 96, 1, 1),
    (3, 7, 5, 192, 40, 1, 1),
]


def ids(c):
    return "n{}h{}w{}ci{}co{}k{}s{}".format(*c)


def shape_of(c):
    n, h, w, ci, co, k, s = c
    return ConvShape(n, h, w, ci, co, k, k, s, s, k // 2, k // 2)


@pytest.mark.parametrize("ci", range(len(CONV_CASES)), ids=[ids(c) for c in CONV_CASES])
def test_conv_fwd_and_stats(ci):
    c = CONV_CASES[ci]
    s = shape_of(c)
    inp = Inputs(100, ci)
    xb, wb = inp.normal(s.x_shape, synth.T_X), inp.weight(s.co, s.kh, s.ci)
    blk = blocks.ConvBlock(s.n, s.h, s.w, s.ci, s.co, s.kh, s.sh)
    x, w = blocks.dev_bf16(xb), blocks.dev_bf16(wb)
    y = torch.empty(s.y_shape, dtype=torch.bfloat16, device="cuda")
    stats = torch.empty(2 * s.co, dtype=torch.float32, device="cuda")
    nb.numbat_conv_fwd(blk.prob, x, w, y, stats, blocks.workspace(blk.ws_fwd))
    torch.cuda.synchronize()
    yref = oracle.conv_fwd(f64(xb), f64(wb), s)
    assert_close(blocks.host_f64(y), yref, "y")
    mref, vref = oracle.bn_stats(yref)
    st = blocks.host_f64(stats)
    assert_stats(st[:s.co], st[s.co:], mref, vref, EPS, "fused batch stats")
    # without statistics y is identical and no workspace is needed
    y2 = torch.empty_like(y)
    nb.numbat_conv_fwd(blk.prob, x, w, y2, None, None)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


@pytest.mark.parametrize("ci", range(len(CONV_CASES)), ids=[ids(c) for c in CONV_CASES])
def test_conv_dgrad(ci):
    c = CONV_CASES[ci]
    s = shape_of(c)
    inp = Inputs(101, ci)
    dyb, wb = inp.normal(s.y_shape, synth.T_DY), inp.weight(s.co, s.kh, s.ci)
    blk = blocks.ConvBlock(s.n, s.h, s.w, s.ci, s.co, s.kh, s.sh)
    dx = torch.full(s.x_shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = blocks.workspace(blk.ws_dgrad)
    nb.numbat_conv_bwd_data(blk.prob, blocks.dev_bf16(dyb), blocks.dev_bf16(wb), dx, False, ws)
    torch.cuda.synchronize()
    ref = oracle.conv_dgrad(f64(dyb), f64(wb), s)
    assert_close(blocks.host_f64(dx), ref, "dx")
    # accumulate into an existing gradient
    x0 = inp.normal(s.x_shape, synth.T_X)
    dxa = blocks.dev_bf16(x0)
    nb.numbat_conv_bwd_data(blk.prob, blocks.dev_bf16(dyb), blocks.dev_bf16(wb), dxa, True, ws)
    torch.cuda.synchronize()
    assert_close(blocks.host_f64(dxa), ref + f64(x0), "dx accumulate")


@pytest.mark.parametrize("ci", range(len(CONV_CASES)), ids=[ids(c) for c in CONV_CASES])
def test_conv_wgrad(ci):
    c = CONV_CASES[ci]
    s = shape_of(c)
    inp = Inputs(102, ci)
    xb, dyb = inp.normal(s.x_shape, synth.T_X), inp.normal(s.y_shape, synth.T_DY)
    blk = blocks.ConvBlock(s.n, s.h, s.w, s.ci, s.co, s.kh, s.sh)
    dw = torch.full(s.w_shape, float("nan"), dtype=torch.float32, device="cuda")
    ws = blocks.workspace(blk.ws_wgrad)
    nb.numbat_conv_bwd_weight(blk.prob, blocks.dev_bf16(xb), blocks.dev_bf16(dyb), dw, False, ws)
    torch.cuda.synchronize()
    ref = oracle.conv_wgrad(f64(xb), f64(dyb), s)
    assert_close(blocks.host_f64(dw), ref, "dw")
    w0 = np.random.default_rng(ci).standard_normal(s.w_shape).astype(np.float32)
    dwa = torch.from_numpy(w0).cuda()
    nb.numbat_conv_bwd_weight(blk.prob, blocks.dev_bf16(xb), blocks.dev_bf16(dyb), dwa, True, ws)
    torch.cuda.synchronize()
    assert_close(blocks.host_f64(dwa), ref + w0.astype(np.float64), "dw accumulate")


def test_conv_strided_views():
    """x and y as channel slices of wider tensors (pixel stride > channels)."""
    s = ConvShape(2, 14, 14, 48, 48, 3, 3, 1, 1, 1, 1)
    inp = Inputs(103)
    big = inp.normal((2, 14, 14, 144), synth.T_X)
    wb = inp.weight(48, 3, 48)
    blk = blocks.ConvBlock(2, 14, 14, 48, 48, 3, 1, x_pixel_stride=144, y_pixel_stride=96)
    xbig = blocks.dev_bf16(big)
    ybig = torch.zeros((2, 14, 14, 96), dtype=torch.bfloat16, device="cuda")
    nb.numbat_conv_fwd(blk.prob, xbig[..., 48:96], blocks.dev_bf16(wb), ybig[..., 40:88])
    torch.cuda.synchronize()
    yref = oracle.conv_fwd(f64(big[..., 48:96]), f64(wb), s)
    got = blocks.host_f64(ybig)
    assert_close(got[..., 40:88], yref, "y view")
    assert np.all(got[..., :40] == 0) and np.all(got[..., 88:] == 0)
    # data gradient into a slice, weight gradient from slices
    dyb = inp.normal((2, 14, 14, 96), synth.T_DY)
    dxbig = torch.zeros((2, 14, 14, 144), dtype=torch.bfloat16, device="cuda")
    ws = blocks.workspace(blk.ws_bytes())
    nb.numbat_conv_bwd_data(blk.prob, blocks.dev_bf16(dyb)[..., 40:88], blocks.dev_bf16(wb), dxbig[..., 48:96], False, ws)
    dw = torch.empty((48, 3, 3, 48), dtype=torch.float32, device="cuda")
    nb.numbat_conv_bwd_weight(blk.prob, xbig[..., 48:96], blocks.dev_bf16(dyb)[..., 40:88], dw, False, ws)
    torch.cuda.synchronize()
    gx = blocks.host_f64(dxbig)
    assert_close(gx[..., 48:96], oracle.conv_dgrad(f64(dyb[..., 40:88]), f64(wb), s), "dx view")
    assert np.all(gx[..., :48] == 0) and np.all(gx[..., 96:] == 0)
    assert_close(blocks.host_f64(dw), oracle.conv_wgrad(f64(big[..., 48:96]), f64(dyb[..., 40:88]), s), "dw views")


def test_conv_strided_views_large():
    """Channel slices at more than 32768 rows (batch 8 at 80x80: the large-tile kernel
    variants): the forward with statistics into a 96-channel slice of a 384-wide buffer from
    a slice of a 192-wide one, the data gradient accumulated into a slice, the weight
    gradient from slices -- as in a C2f block at the detector's batch."""
    n, h, c = 8, 80, 96
    s = ConvShape(n, h, h, c, c, 3, 3, 1, 1, 1, 1)
    inp = Inputs(108)
    xbig = inp.normal((n, h, h, 192), synth.T_X)
    wb = inp.weight(c, 3, c)
    dybig = inp.normal((n, h, h, 384), synth.T_DY)
    dx0 = inp.normal((n, h, h, 192), synth.T_RES)
    blk = blocks.ConvBlock(n, h, h, c, c, 3, 1, x_pixel_stride=192, y_pixel_stride=384)
    x, w = blocks.dev_bf16(xbig), blocks.dev_bf16(wb)
    ybig = torch.zeros((n, h, h, 384), dtype=torch.bfloat16, device="cuda")
    stats = torch.empty(2 * c, dtype=torch.float32, device="cuda")
    ws = blocks.workspace(blk.ws_bytes())
    nb.numbat_conv_fwd(blk.prob, x[..., 96:], w, ybig[..., 192:288], stats, ws)
    dy = blocks.dev_bf16(dybig)
    dxbig = blocks.dev_bf16(dx0)
    nb.numbat_conv_bwd_data(blk.prob, dy[..., 288:], w, dxbig[..., 96:], True, ws)
    dw = torch.empty((c, 3, 3, c), dtype=torch.float32, device="cuda")
    nb.numbat_conv_bwd_weight(blk.prob, x[..., 96:], dy[..., 288:], dw, False, ws)
    torch.cuda.synchronize()
    xs = f64(xbig[..., 96:])
    yref = oracle.conv_fwd(xs, f64(wb), s)
    got = blocks.host_f64(ybig)
    assert_close(got[..., 192:288], yref, "y view")
    assert np.all(got[..., :192] == 0) and np.all(got[..., 288:] == 0)
    mref, vref = oracle.bn_stats(yref)
    st = blocks.host_f64(stats)
    assert_stats(st[:c], st[c:], mref, vref, EPS, "batch stats of a view")
    gx = blocks.host_f64(dxbig)
    dxref = oracle.conv_dgrad(f64(dybig[..., 288:]), f64(wb), s) + f64(dx0[..., 96:])
    assert_close(gx[..., 96:], dxref, "dx accumulated into a view")
    assert np.array_equal(gx[..., :96], f64(dx0[..., :96]))
    assert_close(blocks.host_f64(dw), oracle.conv_wgrad(xs, f64(dybig[..., 288:]), s), "dw from views")


# (400000, 48) and the next two exceed 512 reduce blocks; (3000000, 48) and (250000, 576) meet the
# block cap; then the detector's 20/40/80-wide shapes, the smallest m and the widest c
BN_CASES = [(1000, 8), (4097, 48), (2048, 96), (777, 576), (300, 64), (400000, 48), (3000000, 48), (250000, 576),
            (6400, 576), (25600, 192), (102400, 96), (2, 8), (4, 2048)]


@pytest.mark.parametrize("m,c", BN_CASES)
def test_bn_silu_fwd_given_and_standalone_stats(m, c):
    inp = Inputs(104, c)
    yb = inp.normal((m, c), synth.T_Y, 0.3, 2.0)
    gamma = inp.f32_uniform((c,), synth.T_GAMMA, 0.5, 1.5)
    beta = inp.f32_normal((c,), synth.T_BETA, 0.0, 0.3)
    mean_in = inp.f32_normal((c,), synth.T_MEAN, 0.0, 0.5)
    var_in = inp.f32_uniform((c,), synth.T_VAR, 0.5, 2.0)
    p = nb.bn_problem(m, c, EPS, 0.1)
    y = blocks.dev_bf16(yb)
    out = torch.empty_like(y)
    sm = torch.empty(c, device="cuda")
    sr = torch.empty(c, device="cuda")
    stats = blocks.dev_f32(np.concatenate([mean_in, var_in]))
    g, b = blocks.dev_f32(gamma), blocks.dev_f32(beta)
    nb.numbat_bn_silu_fwd(p, y, stats, g, b, None, out, sm, sr)
    torch.cuda.synchronize()
    ref = oracle.bn_silu_fwd(f64(yb), mean_in.astype(np.float64), var_in.astype(np.float64), gamma.astype(np.float64),
                             beta.astype(np.float64), EPS)
    assert_close(blocks.host_f64(out), ref, "out (given stats)")
    assert np.allclose(blocks.host_f64(sr), 1 / np.sqrt(var_in.astype(np.float64) + EPS), rtol=1e-6)

    # standalone statistics of the bf16 y, plus the running-statistics update
    rm = torch.full((c,), 0.25, device="cuda")
    rv = torch.full((c,), 2.0, device="cuda")
    ws = blocks.workspace(nb.numbat_workspace_size(nb.OP_BN_SILU_FWD, p))
    nb.numbat_bn_silu_fwd(p, y, None, g, b, None, out, sm, sr, rm, rv, ws)
    torch.cuda.synchronize()
    mref, vref = oracle.bn_stats(f64(yb))
    rstd = blocks.host_f64(sr)
    assert_stats(blocks.host_f64(sm), 1 / rstd ** 2 - EPS, mref, vref, EPS, "standalone stats")
    ref = oracle.bn_silu_fwd(f64(yb), mref, vref, gamma.astype(np.float64), beta.astype(np.float64), EPS)
    assert_close(blocks.host_f64(out), ref, "out (standalone stats)")
    rmr, rvr = oracle.running_update(np.full(c, 0.25), np.full(c, 2.0), mref, vref, m, 0.1)
    assert np.allclose(blocks.host_f64(rm), rmr, rtol=1e-5, atol=1e-6)
    assert np.allclose(blocks.host_f64(rv), rvr, rtol=1e-5)


def test_bn_silu_fwd_residual_and_views():
    m, c = 2000, 96
    inp = Inputs(105)
    ybig = inp.normal((m, 192), synth.T_Y)
    rb = inp.normal((m, 96), synth.T_RES)
    gamma = inp.f32_uniform((c,), synth.T_GAMMA, 0.5, 1.5)
    beta = inp.f32_normal((c,), synth.T_BETA, 0.0, 0.3)
    p = nb.bn_problem(m, c, EPS, y_pixel_stride=192, a_pixel_stride=288, r_pixel_stride=96)
    outbig = torch.zeros((m, 288), dtype=torch.bfloat16, device="cuda")
    sm, sr = torch.empty(c, device="cuda"), torch.empty(c, device="cuda")
    ws = blocks.workspace(nb.numbat_workspace_size(nb.OP_BN_SILU_FWD, p))
    nb.numbat_bn_silu_fwd(p, blocks.dev_bf16(ybig)[:, 96:], None, blocks.dev_f32(gamma), blocks.dev_f32(beta),
                          blocks.dev_bf16(rb), outbig[:, 192:], sm, sr, ws=ws)
    torch.cuda.synchronize()
    y = f64(ybig[:, 96:])
    mref, vref = oracle.bn_stats(y)
    ref = oracle.bn_silu_fwd(y, mref, vref, gamma.astype(np.float64), beta.astype(np.float64), EPS, f64(rb))
    got = blocks.host_f64(outbig)
    assert_close(got[:, 192:], ref, "out with residual into a view")
    assert np.all(got[:, :192] == 0)


@pytest.mark.parametrize("m,c", BN_CASES)
def test_bn_silu_bwd(m, c):
    inp = Inputs(106, c)
    yb = inp.normal((m, c), synth.T_Y, -0.2, 1.5)
    gb = inp.normal((m, c), synth.T_G)
    r0 = inp.normal((m, c), synth.T_RES)
    gamma = inp.f32_uniform((c,), synth.T_GAMMA, 0.5, 1.5)
    beta = inp.f32_normal((c,), synth.T_BETA, 0.0, 0.3)
    p = nb.bn_problem(m, c, EPS)
    y = blocks.dev_bf16(yb)
    ga, be = blocks.dev_f32(gamma), blocks.dev_f32(beta)
    out = torch.empty_like(y)
    sm, sr = torch.empty(c, device="cuda"), torch.empty(c, device="cuda")
    ws = blocks.workspace(max(nb.numbat_workspace_size(nb.OP_BN_SILU_FWD, p),
                              nb.numbat_workspace_size(nb.OP_BN_SILU_BWD, p)))
    nb.numbat_bn_silu_fwd(p, y, None, ga, be, None, out, sm, sr, ws=ws)
    dy = torch.empty_like(y)
    dg, db = torch.empty(c, device="cuda"), torch.empty(c, device="cuda")
    rg = blocks.dev_bf16(r0)
    nb.numbat_bn_silu_bwd(p, blocks.dev_bf16(gb), y, sm, sr, ga, be, dy, dg, db, rg, ws=ws)
    torch.cuda.synchronize()
    mref, vref = oracle.bn_stats(f64(yb))
    dyr, dgr, dbr = oracle.bn_silu_bwd(f64(gb), f64(yb), mref, vref, gamma.astype(np.float64),
                                       beta.astype(np.float64), EPS)
    assert_close(blocks.host_f64(dy), dyr, "dy")
    assert_close(blocks.host_f64(dg), dgr, "dgamma")
    assert_close(blocks.host_f64(db), dbr, "dbeta")
    assert_close(blocks.host_f64(rg), f64(r0) + f64(gb), "residual grad")
    # the workspace's counter header is left zero
    assert int(ws[:256].count_nonzero()) == 0
    # bitwise reproducible (whichever path the layer takes)
    dy2, dg2, db2 = torch.empty_like(dy), torch.empty_like(dg), torch.empty_like(db)
    nb.numbat_bn_silu_bwd(p, blocks.dev_bf16(gb), y, sm, sr, ga, be, dy2, dg2, db2, None, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(dy, dy2) and torch.equal(dg, dg2) and torch.equal(db, db2)


@pytest.mark.parametrize("c", [(4, 20, 20, 96, 96, 3, 1), (4, 20, 20, 288, 288, 3, 1)])
def test_bitwise_determinism(c):
    """Two runs of a block's forward and backward are bit for bit equal."""
    s = shape_of(c)
    inp = Inputs(107)
    xb, wb, gb = inp.normal(s.x_shape, synth.T_X), inp.weight(s.co, 3, s.ci), inp.normal(s.y_shape, synth.T_G)
    blk = blocks.ConvBlock(s.n, s.h, s.w, s.ci, s.co, 3, 1)
    x, w, g = blocks.dev_bf16(xb), blocks.dev_bf16(wb), blocks.dev_bf16(gb)
    ga = torch.ones(s.co, device="cuda")
    be = torch.zeros(s.co, device="cuda")
    runs = []
    for _ in range(2):
        f = blk.forward(x, w, ga, be)
        b = blk.backward(g, x, w, ga, be, f)
        torch.cuda.synchronize()
        runs.append({**{k: v.clone() for k, v in f.items()}, **{k: v.clone() for k, v in b.items()}})
    for k in runs[0]:
        assert torch.equal(runs[0][k], runs[1][k]), k
