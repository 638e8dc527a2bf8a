"""A Conv+BN+SiLU forward+backward sequence captured into a HIP graph replays to the
eager result, bitwise, on every replay (eager work between replays)."""
import pytest

from parity import Inputs
from paper_2609_10632_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    from paper_2609_10632_amd import blocks


def test_graph_replay_matches_eager():
    specs = [(4, 40, 48, 96, 3, 2), (4, 20, 96, 96, 3, 1), (4, 20, 96, 64, 1, 1)]
    layers = []
    for i, (n, h, ci, co, k, s) in enumerate(specs):
        ip = Inputs(200, i)
        blk = blocks.ConvBlock(n, h, h, ci, co, k, s)
        x = blocks.dev_bf16(ip.normal((n, h, h, ci), synth.T_X))
        w = blocks.dev_bf16(ip.weight(co, k, ci))
        g = blocks.dev_bf16(ip.normal((n, blk.ho, blk.ho, co), synth.T_G))
        ga = torch.ones(co, device="cuda")
        be = torch.zeros(co, device="cuda")
        ws = blocks.workspace(blk.ws_bytes())
        fwd = {"y": torch.empty((n, blk.ho, blk.ho, co), dtype=torch.bfloat16, device="cuda")}
        fwd["a"] = torch.empty_like(fwd["y"])
        layers.append(dict(blk=blk, x=x, w=w, g=g, ga=ga, be=be, ws=ws, fwd=fwd, out={}))

    from paper_2609_10632_amd import numbat as nb

    def step():
        for L in layers:
            b = L["blk"]
            L.setdefault("stats", torch.empty(2 * b.co, device="cuda"))
            L.setdefault("sm", torch.empty(b.co, device="cuda"))
            L.setdefault("sr", torch.empty(b.co, device="cuda"))
            nb.numbat_conv_fwd(b.prob, L["x"], L["w"], L["fwd"]["y"], L["stats"], L["ws"])
            nb.numbat_bn_silu_fwd(b.bn(), L["fwd"]["y"], L["stats"], L["ga"], L["be"], None, L["fwd"]["a"], L["sm"],
                                  L["sr"], ws=L["ws"])
        for L in reversed(layers):
            b = L["blk"]
            o = L["out"]
            o.setdefault("dy", torch.empty_like(L["fwd"]["y"]))
            o.setdefault("dg", torch.empty(b.co, device="cuda"))
            o.setdefault("db", torch.empty(b.co, device="cuda"))
            o.setdefault("dw", torch.empty((b.co, b.k, b.k, b.ci), device="cuda"))
            o.setdefault("dx", torch.empty_like(L["x"]))
            nb.numbat_bn_silu_bwd(b.bn(), L["g"], L["fwd"]["y"], L["sm"], L["sr"], L["ga"], L["be"], o["dy"], o["dg"],
                                  o["db"], None, ws=L["ws"])
            nb.numbat_conv_bwd_weight(b.prob, L["x"], o["dy"], o["dw"], False, L["ws"])
            nb.numbat_conv_bwd_data(b.prob, o["dy"], L["w"], o["dx"], False, L["ws"])

    step()
    torch.cuda.synchronize()
    outs = [L["fwd"]["a"] for L in layers] + [t for L in layers for t in L["out"].values()] + \
           [L["stats"] for L in layers]
    ref = [t.clone() for t in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(4):
        for t in outs:
            t.fill_(float("nan"))
        # unrelated eager work between replays
        torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (t, r) in enumerate(zip(outs, ref)):
            assert torch.equal(t, r), f"replay {rep}: output {i} differs"
