"""GPU parity of the SPPF max pool and the neck's nearest 2x upsampling against the fp64
oracle.  Index work is compared bit for bit: pooled values (bf16 maxima are exact) and the
stored first-maximum positions, including inputs full of ties; the upsampled copy is exact.
Gradients (fp32 sums of bf16 values, rounded once) within rel_inf 2e-2.  Operands are
channel slices of wider buffers, as in the SPPF concatenation."""
import numpy as np
import pytest

from oracle import pool
from parity import Inputs, assert_close, f64, report
from paper_2609_10632_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    from paper_2609_10632_amd import blocks
    from paper_2609_10632_amd import numbat as nb


@pytest.mark.parametrize("ties", [False, True])
@pytest.mark.parametrize("shape", [(16, 20, 20, 288), (2, 7, 9, 16), (1, 1, 3, 8)])
def test_maxpool(shape, ties):
    n, h, w, c = shape
    ip = Inputs(130, c + ties)
    big = ip.normal((n, h, w, 4 * c), synth.T_X)
    if ties:  # few distinct values: most windows hold several equal maxima
        big = synth.f64_to_bf16_bits(np.floor(f64(big) * 1.5))
    dyb = ip.normal((n, h, w, 2 * c), synth.T_DY)
    x = blocks.dev_bf16(big)
    ybig = torch.zeros((n, h, w, 4 * c), dtype=torch.bfloat16, device="cuda")
    idx = torch.full((n, h, w, c), 255, dtype=torch.uint8, device="cuda")
    p = nb.pool_problem(n, h, w, c, x_pixel_stride=4 * c, y_pixel_stride=4 * c)
    nb.numbat_maxpool5_fwd(p, x[..., :c], ybig[..., c:2 * c], idx)
    pb = nb.pool_problem(n, h, w, c, x_pixel_stride=4 * c, y_pixel_stride=2 * c)
    dx0 = ip.normal((n, h, w, 4 * c), synth.T_RES)
    dxbig = blocks.dev_bf16(dx0)
    nb.numbat_maxpool5_bwd(pb, blocks.dev_bf16(dyb)[..., c:], idx, dxbig[..., :c], True)
    torch.cuda.synchronize()
    yref, iref = pool.maxpool_fwd(f64(big[..., :c]))
    got = blocks.host_f64(ybig)
    assert np.array_equal(got[..., c:2 * c], yref), "pooled values"
    assert np.all(got[..., :c] == 0) and np.all(got[..., 2 * c:] == 0)
    assert np.array_equal(idx.cpu().numpy().astype(np.int64), iref), "first-maximum positions"
    dref = pool.maxpool_bwd(f64(dyb[..., c:]), iref) + f64(dx0[..., :c])
    gx = blocks.host_f64(dxbig)
    e = assert_close(gx[..., :c], dref, "max pool dx (accumulated)")
    assert np.array_equal(gx[..., c:], f64(dx0[..., c:]))
    report(f"maxpool {shape} ties={ties}: y and positions bit-exact, dx complete rel_inf {e:.1e}")


@pytest.mark.parametrize("shape", [(16, 20, 20, 576), (16, 40, 40, 384), (3, 5, 7, 8)])
def test_upsample(shape):
    n, h, w, c = shape
    ip = Inputs(131, c)
    xbig = ip.normal((n, h, w, c + 8), synth.T_X)
    ybig = torch.zeros((n, 2 * h, 2 * w, c + 64), dtype=torch.bfloat16, device="cuda")
    p = nb.pool_problem(n, h, w, c, x_pixel_stride=c + 8, y_pixel_stride=c + 64)
    nb.numbat_upsample2x_fwd(p, blocks.dev_bf16(xbig)[..., 8:], ybig[..., 64:])
    dyb = ip.normal((n, 2 * h, 2 * w, c + 64), synth.T_DY)
    d0 = ip.normal((n, h, w, c + 8), synth.T_RES)
    dx = blocks.dev_bf16(d0)
    nb.numbat_upsample2x_bwd(p, blocks.dev_bf16(dyb)[..., 64:], dx[..., 8:], True)
    torch.cuda.synchronize()
    got = blocks.host_f64(ybig)
    assert np.array_equal(got[..., 64:], pool.upsample2x_fwd(f64(xbig[..., 8:]))), "upsampled copy"
    assert np.all(got[..., :64] == 0)
    gx = blocks.host_f64(dx)
    e = assert_close(gx[..., 8:], pool.upsample2x_bwd(f64(dyb[..., 64:])) + f64(d0[..., 8:]), "upsample dx")
    assert np.array_equal(gx[..., :8], f64(d0[..., :8]))
    report(f"upsample {shape}: y bit-exact, dx complete rel_inf {e:.1e}")
