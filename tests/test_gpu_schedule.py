"""The benchmarked step schedule computes exactly what the serial step computes.

The benchmark times a two-stream step (each layer's weight gradient on a side stream, enqueued
in groups behind one cross-stream wait, the last layers one by one) replayed from a HIP graph.
Every kernel and every reduction order is the same as in the serial step on one stream, so
every output of every layer must be bitwise equal: forward output, activation, batch
statistics, saved mean/rstd, BN backward output, dgamma, dbeta, data and weight gradients.
Checked for the eager two-stream step (grouped and immediate enqueue) and for three graph
replays, each after filling every output with NaN.
"""
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

from paper_2609_10632_amd import workloads  # noqa: E402

# configuration-4 layers covering every kernel family: the image layer, stride-2 3x3,
# 1x1 on several widths, 3x3 stride 1 at 160/80/40/20, the SPPF and neck convs
NAMES = ["b0", "b1", "b2.cv1", "b2.m0.cv1", "b3", "b4.m0.cv2", "b5", "b6.cv2", "b7", "b8.m0.cv1", "b9.cv1",
         "n15.cv1", "n16", "n21.cv2"]


def snapshot(cs):
    return {(l.name, k): t.clone() for l in cs.layers for k, t in l.outputs().items()}


def fill_nan(cs):
    for l in cs.layers:
        for k, t in l.outputs().items():
            t.fill_(float("nan"))
    torch.cuda.synchronize()


def compare(cs, ref, what):
    now = {(l.name, k): t for l in cs.layers for k, t in l.outputs().items()}
    bad = [f"{n}.{k}" for (n, k), r in ref.items() if not torch.equal(now[(n, k)], r)]
    assert not bad, f"{what}: outputs differ from the serial step: {bad}"


def test_two_stream_step_matches_serial_bitwise():
    from paper_2609_10632_amd.schedule import ConvSet

    wl = workloads.workload(4)
    specs = [l for l in wl.layers if l.name in NAMES]
    cs = ConvSet(specs, wl.n, wl.index, wl.eps, layer_index=[wl.layers.index(l) for l in specs])
    print(f"schedule parity: {len(specs)} layers at batch {wl.n}", flush=True)
    cs.step(overlap=False)
    torch.cuda.synchronize()
    ref = snapshot(cs)
    for defer, group, tail in ((True, 2, 3), (True, 3, 2), (False, 1, 0)):
        fill_nan(cs)
        cs.step(overlap=True, defer=defer, group=group, tail=tail)
        torch.cuda.synchronize()
        compare(cs, ref, f"eager two-stream (defer={defer}, group={group}, tail={tail})")
    # the benchmark's default schedule captured into a graph, replayed three times
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        cs.step(overlap=True)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cs.step(overlap=True)
    torch.cuda.synchronize()
    for rep in range(3):
        fill_nan(cs)
        graph.replay()
        torch.cuda.synchronize()
        compare(cs, ref, f"graph replay {rep}")
        # eager work between replays
        cs.step(overlap=False)
        torch.cuda.synchronize()
        compare(cs, ref, f"eager serial step after replay {rep}")


def test_fused_backward_step_matches_unfused_bitwise():
    """With the BN + SiLU backward formed inside the 3x3 stride-1 layers' data gradients
    (fuse_bwd), every output of every layer equals the unfused serial step's bit for bit:
    serial, two-stream, and graph-replayed (the weight gradients read the dy the fused data
    gradients wrote)."""
    from paper_2609_10632_amd.schedule import ConvSet

    wl = workloads.workload(4)
    specs = [l for l in wl.layers if l.name in NAMES]
    idx = [wl.layers.index(l) for l in specs]
    ref_set = ConvSet(specs, wl.n, wl.index, wl.eps, layer_index=idx)
    ref_set.step(overlap=False)
    torch.cuda.synchronize()
    ref = snapshot(ref_set)
    del ref_set
    cs = ConvSet(specs, wl.n, wl.index, wl.eps, layer_index=idx, fuse_bwd=True)
    fused = [l.name for l in cs.layers if l.fused]
    print(f"fused backward parity: {len(specs)} layers, {len(fused)} fused: {fused}", flush=True)
    assert len(fused) >= 3
    for overlap in (False, True):
        fill_nan(cs)
        cs.step(overlap=overlap)
        torch.cuda.synchronize()
        compare(cs, ref, f"fused backward, two streams={overlap}")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        cs.step(overlap=True)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cs.step(overlap=True)
    torch.cuda.synchronize()
    for rep in range(2):
        fill_nan(cs)
        graph.replay()
        torch.cuda.synchronize()
        compare(cs, ref, f"fused backward graph replay {rep}")
