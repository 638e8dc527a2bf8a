"""GPU parity of the chain-mode network (backbone + neck with the real dataflow: C2f concat
views, residuals, SPPF max pools, nearest upsampling, neck concatenations, gradient fan-in)
against the fp64 oracle, stage-isolated: every operation of one training step is compared
with the oracle's on the GPU's own inputs to that operation, and every gradient buffer with
the oracle's sum of all its contributions (data gradients, residual gradients, upsample and
max-pool backwards, the outputs' upstream gradients).  That checks every connection of the
network -- views, concat offsets, accumulation flags -- while bf16 rounding of intermediate
activations cannot accumulate over the network's depth.

The benchmarked step runs the weight gradients on a second stream; it is first checked bit
for bit against the same step on one stream (every layer's dw, dgamma, dbeta, y and the
image gradient), then the two-stream step's results are compared with the oracle.

Tolerances: rel_inf <= 2e-2 for every bf16 output and gradient; batch statistics 1e-5;
pooled values, first-maximum positions and upsampled copies bit for bit.  The end-to-end
distance of the three outputs from the oracle's (run from the same seeded input, so bf16
rounding compounds through ~60 layers) is printed, not asserted.

Batch 1 at a 320 x 320 input (P5 is 10 x 10)."""
import numpy as np
import pytest

import oracle
from oracle import ConvShape
from oracle import detector as odet
from oracle import pool
from parity import assert_close, assert_stats, f64, rel_inf, report

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    from paper_2609_10632_amd import blocks
    from paper_2609_10632_amd.detector import Detector

EPS = 1e-3
H = blocks.host_f64 if torch.cuda.is_available() else None


def base_and_offset(t):
    """The whole NHWC buffer a channel-slice view belongs to, and the view's first channel."""
    b = t._base if t._base is not None else t
    return b, (t.data_ptr() - b.data_ptr()) // t.element_size()


@pytest.mark.parametrize("affine", [False, True])
def test_chain_network_stage_isolated(affine):
    n, hin = 1, 320
    det = Detector(n, hin, EPS)
    host, xb, gs = det.seeded(40, affine=affine)
    print(f"chain network n={n} input {hin}: GPU step on one stream", flush=True)
    det.step(overlap=False)
    torch.cuda.synchronize()
    keys = lambda: {**{(c.name, k): getattr(c, k).clone() for c in det.layers for k in ("dw", "dgamma", "dbeta", "y")},
                    ("image", "dx"): det.dx.clone()}
    serial = keys()
    print("GPU step, weight gradients on the side stream", flush=True)
    det.step()
    torch.cuda.synchronize()
    now = keys()
    bad = [k for k in serial if not torch.equal(serial[k], now[k])]
    assert not bad, f"two-stream step differs from the serial one: {bad[:5]}"
    print("oracle, stage by stage", flush=True)
    W = {k: (f64(w), g.astype(np.float64), b.astype(np.float64)) for k, (w, g, b) in host.items()}
    contrib = {}  # gradient buffer -> (buffer, expected sum of every contribution to its channels)

    def add(t, v):
        b, off = base_and_offset(t)
        if b.data_ptr() not in contrib:
            contrib[b.data_ptr()] = (b, np.zeros(tuple(b.shape)))
        contrib[b.data_ptr()][1][..., off:off + t.shape[-1]] += v

    worst = {"fwd": 0.0, "bwd": 0.0}
    for g_init, t in zip(gs, (det.g3, det.g4, det.g5)):
        add(t, f64(g_init))
    for op in det.ops:
        if op[0] == "pool":
            _, pp, src, dst, idx, ddst, dsrc = op
            yref, iref = pool.maxpool_fwd(H(src))
            assert np.array_equal(H(dst), yref) and np.array_equal(idx.cpu().numpy().astype(np.int64), iref)
            add(dsrc, pool.maxpool_bwd(H(ddst), iref))
            continue
        if op[0] == "up":
            _, pp, src, dst, ddst, dsrc = op
            assert np.array_equal(H(dst), pool.upsample2x_fwd(H(src)))
            add(dsrc, pool.upsample2x_bwd(H(ddst)))
            continue
        c = op[1]
        w, ga, be = W[c.name]
        sp = c.spec
        x = H(c.x)
        s = ConvShape(n, x.shape[1], x.shape[2], sp.ci, sp.co, sp.k, sp.k, sp.s, sp.s, sp.p, sp.p)
        # forward: y, statistics, a (with the GPU's residual input)
        yref = oracle.conv_fwd(x, w, s)
        worst["fwd"] = max(worst["fwd"], assert_close(H(c.y), yref, f"{c.name} y"))
        st = H(c.stats)
        mref, vref = oracle.bn_stats(yref)
        assert_stats(st[:sp.co], st[sp.co:], mref, vref, EPS, f"{c.name} stats")
        res = H(c.res) if c.res is not None else None
        aref = oracle.bn_silu_fwd(yref, mref, vref, ga, be, EPS, res)
        worst["fwd"] = max(worst["fwd"], assert_close(H(c.out), aref, f"{c.name} a"))
        # backward from the GPU's final upstream gradient, its stored y and statistics
        g = H(c.dout)
        dyref, dgref, dbref = oracle.bn_silu_bwd(g, H(c.y), st[:sp.co], st[sp.co:], ga, be, EPS)
        for nm, got, ref in (("dy", c.dy, dyref), ("dgamma", c.dgamma, dgref), ("dbeta", c.dbeta, dbref)):
            worst["bwd"] = max(worst["bwd"], assert_close(H(got), ref, f"{c.name} {nm}"))
        dy = H(c.dy)
        worst["bwd"] = max(worst["bwd"], assert_close(H(c.dw), oracle.conv_wgrad(x, dy, s), f"{c.name} dw"))
        add(c.dx, oracle.conv_dgrad(dy, w, s))
        if c.dres is not None:
            add(c.dres, g)
    for k, (t, ref) in contrib.items():
        worst["bwd"] = max(worst["bwd"], assert_close(H(t), ref, f"gradient buffer {tuple(t.shape)}"))
    # end to end (diagnostic): the oracle network from the same seeded input
    st = odet.forward(f64(xb), W, EPS)
    e2e = {nm: rel_inf(H(t), st[nm]) for nm, t in (("P3", det.p3), ("P4", det.p4), ("P5", det.p5))}
    report(f"chain network n={n} input {hin} affine={affine}: every op stage-isolated (65 convs: y, stats, a, dy, "
           f"dgamma, dbeta, dw; 3 max pools and 2 upsamples bit-exact; {len(contrib)} gradient buffers as sums of "
           f"their contributions) worst rel_inf fwd {worst['fwd']:.1e} bwd {worst['bwd']:.1e}; end to end "
           + " ".join(f"{k} {v:.1e}" for k, v in e2e.items()))
