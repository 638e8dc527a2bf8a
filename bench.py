#!/usr/bin/env python3
"""Benchmark of the Conv2d + BN(train) + SiLU hot path on one MI355X.

Workload (default): the 65 Conv+BN+SiLU layers of the YOLOv8m-class backbone and
neck at batch 16, 640x640 input (the detector of the paper's case study, Sec. 6.1,
per-GPU batch 16 of Table 1), in set mode: every layer is an independent problem
with seeded inputs x ~ N(0,1) (bf16), Kaiming-uniform weights, gamma = 1, beta = 0,
upstream gradient g ~ N(0,1).  One step = forward over the layers in network order
(conv_fwd with fused batch statistics, bn_silu_fwd), then backward in reverse order
(bn_silu_bwd, conv_bwd_weight, conv_bwd_data) -- every row of the hot path.

Prints ONE JSON line.  value = conv FLOPs of the step (fwd + dgrad + wgrad,
2*M*N*K each) / measured step time, in TFLOP/s; the step is captured once into a HIP
graph (replays are checked bitwise against the eager step) and replayed K times.
roofline = the dominant conv kernel's algorithmic FLOPs / its summed launch durations,
from HIP events the library records around every kernel on its launch stream during K
further (eager) steps.  cpu_baseline = the fp64 oracle on a bounded sample (all layers
at batch 2), on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4, help="workload configuration (4 or 5)")
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-events", action="store_true", help="skip the instrumented (per-kernel timing) steps")
    ap.add_argument("--no-graph", action="store_true", help="time eager launches instead of a HIP graph replay")
    ap.add_argument("--streams", type=int, default=2, choices=(1, 2),
                    help="1: the whole step on one stream; 2 (default): each layer's weight gradient on a "
                         "second stream once its data gradient is done, overlapping the next layers' "
                         "latency-bound BN backward")
    ap.add_argument("--serial", action="store_true", help="same as --streams 1")
    ap.add_argument("--wgrad-order", choices=("deferred", "immediate"), default="deferred",
                    help="two streams: enqueue layer L's weight gradient after layer L-1's BN backward "
                         "(deferred, default) or right after layer L's data gradient (immediate)")
    ap.add_argument("--wgrad-group", type=int, default=1,
                    help="deferred order: enqueue the weight gradients in groups of this many layers behind "
                         "one cross-stream wait (each wait costs the main queue a completion signal)")
    ap.add_argument("--wgrad-tail", type=int, default=0,
                    help="the last this many layers of the backward pass are enqueued one by one")
    ap.add_argument("--fuse-bwd", action="store_true",
                    help="the 3x3 stride-1 layers form dy inside their data gradient (the BN + SiLU backward "
                         "prologue) instead of a separate BN backward apply pass; slower on this GPU, off by "
                         "default")
    ap.add_argument("--layers", type=str, default=None, help="comma-separated layer names (subset)")
    ap.add_argument("--detail", type=str, default=None,
                    help="write per-layer x pass timings (JSON) to this file, and a markdown table beside it")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the extra measurements (chain mode, optimiser step, configuration 5, cold-cache "
                         "steps, copy bandwidth)")
    return ap.parse_args()


class SclkSampler:
    """Samples the GPU's current shader clock (the starred level of pp_dpm_sclk) every 20 ms on
    a host thread while active; mean / min / max in MHz."""

    def __init__(self):
        import glob
        import threading

        paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = paths[0] if paths else None
        self.samples = []
        self._stop = threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True) if self.path else None

    def _read(self):
        try:
            for line in open(self.path):
                if line.strip().endswith("*"):
                    return float(line.split(":")[1].strip().split("Mhz")[0].split("MHz")[0])
        except (OSError, ValueError, IndexError):
            return None
        return None

    def _run(self):
        while not self._stop.wait(0.02):
            v = self._read()
            if v is not None:
                self.samples.append(v)

    def __enter__(self):
        if self._t:
            self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self._t:
            self._t.join()

    def summary(self):
        if not self.samples:
            return None
        v = self.samples
        return {"mean_mhz": round(sum(v) / len(v), 1), "min_mhz": min(v), "max_mhz": max(v), "samples": len(v)}


def hbm_copy_gbs(torch, nbytes=1 << 30, reps=10):
    """Device-to-device copy of nbytes (read + write counted), GB/s: the achievable HBM figure."""
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2 * nbytes * reps / (e0.elapsed_time(e1) / 1e3) / 1e9
    del a, b
    return round(gbs, 1)


def graph_of(torch, step):
    """Capture one step (after a side-stream warm-up) into a HIP graph."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    return g


def time_replays(torch, graph, steps):
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        graph.replay()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def cold_cache_ms(torch, graph, steps, evict_bytes=1 << 30):
    """Median step time with the caches cold: before every timed replay a 1 GiB buffer is
    written (more than the 256 MB Infinity Cache and the L2s hold), outside the events."""
    buf = torch.empty(evict_bytes // 4, dtype=torch.float32, device="cuda")
    times = []
    for i in range(steps):
        buf.fill_(float(i))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    del buf
    times.sort()
    return round(times[len(times) // 2], 3)


def chain_mode(torch, steps, warmup):
    """The 65 layers as one network (real dataflow, SPPF pools, upsampling, concatenations) at
    batch 16, 640 x 640, graph-replayed, the weight gradients on a second stream."""
    from paper_2609_10632_amd.detector import Detector

    det = Detector(16, 640)
    det.seeded(4)
    for _ in range(warmup):
        det.step()
    g = graph_of(torch, det.step)
    ms = time_replays(torch, g, steps)
    out = {"ms_per_step": round(ms, 3), "tflops": round(det.flops / (ms / 1e3) / 1e12, 2),
           "pct_mfma_peak": round(100 * det.flops / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 2),
           "step_gflop": round(det.flops / 1e9, 2), "launch": "hip graph replay", "streams": 2,
           "batch": 16, "input": "640x640"}
    del g, det
    torch.cuda.empty_cache()
    return out


def prologue_fusion(torch, steps):
    """Prologue fusion on the C2f bottleneck convs at batch 16, graph-replayed on one stream.
    fwd: the second conv fed by the first's pre-BN output -- the first's BN + SiLU as its own
    pass (writes the activation) followed by the forward, against the prologue-fused forward
    that forms the activation in the conv's operand staging (both with batch statistics).
    bwd: a conv's BN + SiLU backward (reduce, finalize, apply writing dy) followed by its data
    gradient, against the BN backward without dy followed by the data gradient that forms dy
    in its operand staging and writes it."""
    from paper_2609_10632_amd import blocks
    from paper_2609_10632_amd import numbat as nb

    out = {}
    for name, (n, h, c) in (("b2.m0.cv2", (16, 160, 48)), ("b4.m0.cv2", (16, 80, 96)),
                            ("b6.m0.cv2", (16, 40, 192)), ("b8.m0.cv2", (16, 20, 288))):
        blk = blocks.ConvBlock(n, h, h, c, c, 3, 1)
        g = torch.Generator(device="cuda").manual_seed(7)
        yp = torch.randn((n, h, h, c), device="cuda", generator=g).to(torch.bfloat16)
        w = (torch.randn((c, 3, 3, c), device="cuda", generator=g) * 0.03).to(torch.bfloat16)
        prev = torch.cat([torch.zeros(c, device="cuda"), torch.ones(c, device="cuda")])
        ga, be = torch.ones(c, device="cuda"), torch.zeros(c, device="cuda")
        act = torch.empty_like(yp)
        y = torch.empty((n, h, h, c), dtype=torch.bfloat16, device="cuda")
        st = torch.empty(2 * c, device="cuda")
        sm, sr = torch.empty(c, device="cuda"), torch.empty(c, device="cuda")
        ws = blocks.workspace(blk.ws_fwd)
        bnp = nb.bn_problem(n * h * h, c)

        def unfused():
            nb.numbat_bn_silu_fwd(bnp, yp, prev, ga, be, None, act, sm, sr)
            nb.numbat_conv_fwd(blk.prob, act, w, y, st, ws)

        def fused():
            nb.numbat_conv_fwd_bn_silu_prologue(blk.prob, yp, prev, ga, be, 1e-3, w, y, st, ws)

        gb = torch.randn((n, h, h, c), device="cuda", generator=g).to(torch.bfloat16)
        dy = torch.empty_like(gb)
        dx = torch.empty_like(gb)
        dg, db = torch.empty(c, device="cuda"), torch.empty(c, device="cuda")
        wsb = blocks.workspace(max(blk.ws_dgrad, nb.numbat_workspace_size(nb.OP_BN_SILU_BWD, bnp)))
        nb.numbat_bn_silu_fwd(bnp, yp, None, ga, be, None, act, sm, sr, ws=blocks.workspace(blk.ws_bytes()))

        def unfused_bwd():
            nb.numbat_bn_silu_bwd(bnp, gb, yp, sm, sr, ga, be, dy, dg, db, None, ws=wsb)
            nb.numbat_conv_bwd_data(blk.prob, dy, w, dx, False, wsb)

        def fused_bwd():
            nb.numbat_bn_silu_bwd(bnp, gb, yp, sm, sr, ga, be, None, dg, db, None, ws=wsb)
            nb.numbat_conv_bwd_data_bn_silu_prologue(blk.prob, gb, yp, sm, sr, ga, be, dg, db, w, dx, dy)

        out[name] = {}
        for part, uf, ff in (("fwd", unfused, fused), ("bwd", unfused_bwd, fused_bwd)):
            res = {}
            for k, f in (("unfused_ms", uf), ("fused_ms", ff)):
                for _ in range(3):
                    f()
                gr = graph_of(torch, f)
                res[k] = round(time_replays(torch, gr, max(20, steps)), 4)
                del gr
            res["saved_ms"] = round(res["unfused_ms"] - res["fused_ms"], 4)
            out[name][part] = res
    return out


def optimizer_step(torch, steps):
    """The fused global-norm clip + SGD-Nesterov step over the detector's 243 parameter tensors
    (25.9M fp32 parameters, three groups)."""
    from paper_2609_10632_amd import numbat as nb
    from paper_2609_10632_amd import workloads

    shapes = []
    for l, bn, bias in [(l, True, False) for l in workloads.backbone_neck_layers()] + \
            workloads.faithful_head_param_tensors():
        shapes.append((l.co * l.k * l.k * l.ci, 0))
        if bn:
            shapes += [(l.co, 1), (l.co, 2)]
        if bias:
            shapes.append((l.co, 2))
    total = sum(n for n, _ in shapes)
    w = torch.randn(total, device="cuda") * 0.05
    g = torch.randn(total, device="cuda") * 1e-3
    m = torch.zeros(total, device="cuda")
    ents, pos = [], 0
    for n, grp in shapes:
        pad = (-pos) % 4  # 16-byte aligned tensors
        pos += pad
        ents.append((w[pos:pos + n], g[pos:pos + n], m[pos:pos + n], grp))
        pos += n
    table = torch.frombuffer(bytearray(nb.param_table(ents)), dtype=torch.uint8).cuda()
    ws = torch.zeros(nb.numbat_workspace_size(nb.OP_CLIP_SGD_NESTEROV, nb.bn_problem(2, 8)), dtype=torch.uint8,
                     device="cuda")
    hp = [(0.01, 3.75e-4), (0.01, 0.0), (0.1, 0.0)]
    fn = lambda: nb.numbat_clip_sgd_nesterov(table, len(ents), hp, 0.937, 10.0, None, ws)
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    nbytes = sum(n for n, _ in shapes) * (4 + 20)  # squared-norm pass reads g; the update reads w, g, buf, writes w, buf
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"tensors": len(shapes), "parameters": sum(n for n, _ in shapes), "ms": round(ms, 4),
            "bytes": nbytes, "gbs": round(gbs, 1), "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 3)}


def config_set(torch, cfg, batch, steps, warmup, two=True):
    """Set-mode step of a configuration at a batch (two streams, graph-replayed)."""
    from paper_2609_10632_amd.schedule import ConvSet
    from paper_2609_10632_amd.workloads import workload

    wl = workload(cfg, batch)
    cs = ConvSet(wl.layers, wl.n, wl.index, wl.eps, wl.g_std)
    for _ in range(warmup):
        cs.step(overlap=two)
    g = graph_of(torch, lambda: cs.step(overlap=two))
    ms = time_replays(torch, g, steps)
    flops = sum(3 * l.flops for l in cs.layers)
    out = {"layers": len(cs.layers), "batch": wl.n, "ms_per_step": round(ms, 3),
           "tflops": round(flops / (ms / 1e3) / 1e12, 2),
           "pct_mfma_peak": round(100 * flops / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 2),
           "step_gflop": round(flops / 1e9, 2)}
    del g, cs
    torch.cuda.empty_cache()
    return out


PASSES = ("conv_fwd", "bn_silu_fwd", "bn_silu_bwd", "conv_bwd_weight", "conv_bwd_data")


def write_detail(torch, args, step, layers, wl):
    """Per layer x pass: median of five serial steps' HIP-event times (launch gaps included),
    with each pass's algorithmic work against the roofline that binds it: conv passes 2 M N K
    FLOPs and their operand bytes (fwd x + W + y, dgrad dy + W + dx in bf16, wgrad x + dy in
    bf16 + dW in fp32); BN passes 4 (fwd) and 10 (bwd) bytes per element (a layer whose data
    gradient forms dy: BN backward 4, data gradient g + y + W in, dx + dy out).  JSON to
    args.detail, a markdown table beside it."""
    reps = []
    for _ in range(5):
        ev = {l.name: [torch.cuda.Event(enable_timing=True) for _ in range(7)] for l in layers}
        step(ev, overlap=False)
        torch.cuda.synchronize()
        # (a layer whose data gradient forms dy runs it before the weight gradient)
        pairs = lambda l: ((0, 1), (1, 2), (3, 4), (5, 6), (4, 5)) if l.fused else ((0, 1), (1, 2), (3, 4), (4, 5),
                                                                                     (5, 6))
        reps.append({l.name: [ev[l.name][a].elapsed_time(ev[l.name][b]) for a, b in pairs(l)] for l in layers})
    per_layer = {l.name: [sorted(r[l.name][k] for r in reps)[2] for k in range(5)] for l in layers}
    rows, tot = [], {p: 0.0 for p in PASSES}
    for l in layers:
        sp, blk = l.spec, l.blk
        n = blk.n
        xb = n * sp.h * sp.h * sp.ci * 2
        yb = blk.m * sp.co * 2
        wb = sp.co * sp.k * sp.k * sp.ci * 2
        work = {"conv_fwd": (l.flops, xb + wb + yb), "bn_silu_fwd": (0, 4 * l.bn_elems),
                "bn_silu_bwd": (0, 10 * l.bn_elems), "conv_bwd_weight": (l.flops, xb + yb + 2 * wb),
                "conv_bwd_data": (l.flops, yb + wb + xb)}
        if l.fused:  # BN backward: the reduce (g, y); data gradient: g, y and W in, dx and dy out
            work["bn_silu_bwd"] = (0, 4 * l.bn_elems)
            work["conv_bwd_data"] = (l.flops, 3 * yb + wb + xb)
        for k, pname in enumerate(PASSES):
            ms = per_layer[l.name][k]
            tot[pname] += ms
            fl, by = work[pname]
            tf = fl / (ms / 1e3) / 1e12 if fl else 0.0
            gbs = by / (ms / 1e3) / 1e9
            t_mfma, t_hbm = fl / (PEAK_BF16_TFLOPS * 1e12), by / (PEAK_HBM_GBS * 1e9)
            bound = "mfma" if t_mfma >= t_hbm else "hbm"
            frac = max(t_mfma, t_hbm) / (ms / 1e3)
            rows.append((l.name, pname, ms * 1e3, tf, 100 * tf / PEAK_BF16_TFLOPS, gbs, 100 * gbs / PEAK_HBM_GBS, bound,
                         100 * frac))
    with open(args.detail, "w") as f:
        json.dump({"per_layer_ms": per_layer, "passes": PASSES, "flops": {l.name: l.flops for l in layers}}, f,
                  indent=1)
    md = os.path.splitext(args.detail)[0] + ".md"
    with open(md, "w") as f:
        f.write(f"# Per layer x pass, configuration {wl.index}, batch {wl.n} (serial step, median of 5, HIP events)\n\n")
        f.write("| layer | pass | us | TFLOP/s | % MFMA peak | GB/s | % HBM peak | binding roofline | % of it |\n")
        f.write("|---|---|---|---|---|---|---|---|---|\n")
        for r in rows:
            f.write(f"| {r[0]} | {r[1]} | {r[2]:.1f} | {r[3]:.1f} | {r[4]:.1f} | {r[5]:.0f} | {r[6]:.1f} | {r[7]} | "
                    f"{r[8]:.1f} |\n")
        f.write("\n| pass | ms per step |\n|---|---|\n")
        for pname in PASSES:
            f.write(f"| {pname} | {tot[pname]:.3f} |\n")


# HBM traffic per launch measured with rocprofv3 counters (FETCH_SIZE, WRITE_SIZE, each
# scaled by what it reads for a plain device copy) for a kernel class on one workload; the
# figure is used only while the kernel's sources hash to the value recorded with it.
TRAFFIC_PROFILES = {
    ("wgrad_igemm", 4, 16): ("profiles/wgrad_igemm_c4_b16_traffic.md",
                             ("paper_2609_10632_amd/csrc/conv_wgrad.hip", "paper_2609_10632_amd/csrc/conv_wgrad_halo.hip",
                              "paper_2609_10632_amd/csrc/common.h", "paper_2609_10632_amd/csrc/kernels.h")),
    ("conv_fwd_igemm", 4, 16): ("profiles/conv_fwd_igemm_c4_b16_traffic.md",
                                ("paper_2609_10632_amd/csrc/conv_gemm.hip", "paper_2609_10632_amd/csrc/common.h",
                                 "paper_2609_10632_amd/csrc/kernels.h")),
    ("conv_dgrad_igemm", 4, 16): ("profiles/conv_dgrad_igemm_c4_b16_traffic.md",
                                  ("paper_2609_10632_amd/csrc/conv_gemm.hip", "paper_2609_10632_amd/csrc/conv_aux.hip",
                                   "paper_2609_10632_amd/csrc/common.h", "paper_2609_10632_amd/csrc/kernels.h")),
}


def committed_traffic(kernel_class, config_index, batch):
    import hashlib

    entry = TRAFFIC_PROFILES.get((kernel_class, config_index, batch))
    if entry is None:
        return None
    here = os.path.dirname(os.path.abspath(__file__))
    prof, sources = entry
    try:
        text = open(os.path.join(here, prof)).read()
        h = hashlib.sha256()
        for src in sources:
            with open(os.path.join(here, src), "rb") as f:
                h.update(f.read())
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines() if line.startswith(("kernel_source_sha256", "traffic")))
    if fields.get("kernel_source_sha256", "").strip() != h.hexdigest():
        return None  # the kernel changed since the counters were taken
    return float(fields["traffic_bytes_per_launch"])


def cpu_baseline(wl, threads_hint):
    """The fp64 oracle on a bounded sample of the same workload: every layer at batch 2
    (about 10 s on 16 host threads), forward + BN/SiLU forward and backward + data and
    weight gradients."""
    import numpy as np

    import oracle
    from oracle import ConvShape
    from paper_2609_10632_amd import synth

    oracle.build(force=False)
    flops = 0.0
    t_total = 0.0
    nb = 2
    for idx, l in enumerate(wl.layers):
        sid = lambda t: synth.stream_id(90 + wl.index, idx, t)
        b = synth.kaiming_uniform_bound(l.ci * l.k * l.k)
        x = synth.bf16_to_f64(synth.bf16((nb, l.h, l.h, l.ci), sid(synth.T_X)))
        w = synth.bf16_to_f64(synth.bf16((l.co, l.k, l.k, l.ci), sid(synth.T_W), synth.UNIFORM, -b, b))
        g = synth.bf16_to_f64(synth.bf16((nb, l.ho, l.ho, l.co), sid(synth.T_G)))
        s = ConvShape(nb, l.h, l.h, l.ci, l.co, l.k, l.k, l.s, l.s, l.p, l.p)
        ones, zeros = np.ones(l.co), np.zeros(l.co)
        t0 = time.perf_counter()
        f = oracle.block_fwd(x, w, s, ones, zeros, wl.eps)
        oracle.block_bwd(g, x, w, s, f, ones, zeros, wl.eps)
        t_total += time.perf_counter() - t0
        flops += 3 * l.gemm_flops(nb)
    return {"value": flops / t_total / 1e12, "unit": "TFLOP/s", "cores": threads_hint, "kind": "oracle",
            "sample": f"all {len(wl.layers)} layers at batch {nb} ({nb}/{wl.n} of the step): conv fwd + BN/SiLU fwd/bwd + "
                      f"dgrad + wgrad in fp64; {flops / 1e9:.1f} GFLOP in {t_total:.1f} s"}


def capture_graph(step, check_tensors):
    """Capture one step into a HIP graph; replay it three times, each after an eager fill of
    the checked outputs with NaN, and require every replay to reproduce the eager result
    bitwise.  Returns the graph."""
    import torch

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in check_tensors]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for _ in range(3):
        for t in check_tensors:
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for t, r in zip(check_tensors, ref):
            if not torch.equal(t, r):
                raise RuntimeError("graph replay differs from the eager step")
    return graph


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus}). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_10632_amd import numbat as nb
    from paper_2609_10632_amd.schedule import ConvSet
    from paper_2609_10632_amd.workloads import workload

    nb.load()
    torch.cuda.set_device(0)
    wl = workload(args.config, args.batch)
    specs = wl.layers
    if args.layers:
        want = set(args.layers.split(","))
        specs = [l for l in specs if l.name in want]
    print(f"# setting up {len(specs)} layers of configuration {wl.index} at batch {wl.n}", file=sys.stderr, flush=True)
    cs = ConvSet(specs, wl.n, wl.index, wl.eps, wl.g_std,
                 [wl.layers.index(l) for l in specs], fuse_bwd=args.fuse_bwd)
    layers = cs.layers
    two = args.streams == 2 and not args.serial
    defer = args.wgrad_order == "deferred"
    torch.cuda.synchronize()
    step_flops = sum(3 * l.flops for l in layers)

    def step(ev=None, overlap=True):
        cs.step(ev, overlap=overlap and two, defer=defer, group=args.wgrad_group, tail=args.wgrad_tail)

    print(f"# warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    graph = None
    if not args.no_graph:
        print("# capturing the step into a HIP graph (replays checked bitwise against eager)", file=sys.stderr,
              flush=True)
        probe = [layers[0].dx, layers[0].a, layers[-1].dw, layers[len(layers) // 2].dx, layers[len(layers) // 2].stats,
                 layers[-1].dgamma]
        graph = capture_graph(step, probe)

    # ---- timed region: K steps, nothing else on the stream
    print(f"# timing {args.steps} steps ({'graph replay' if graph else 'eager launches'})", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    with SclkSampler() as sclk:
        t0 = time.perf_counter()
        for _ in range(args.steps):
            if graph is not None:
                graph.replay()
            else:
                step()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    cold = None
    if graph is not None and not args.no_extras:
        print("# cold-cache steps (1 GiB written between replays)", file=sys.stderr, flush=True)
        cold = cold_cache_ms(torch, graph, max(5, args.steps // 2))

    # ---- instrumented region: the same K steps, eager, every kernel bracketed by HIP events on
    # its launch stream (library timing), for the per-kernel roofline
    n_cls = nb.numbat_kernel_class_count()
    per_cls = {}
    ms_instr = None
    if not args.no_events:
        print(f"# instrumented {args.steps} steps (per-kernel HIP events)", file=sys.stderr, flush=True)
        torch.cuda.synchronize()
        nb.numbat_timing_enable(True)
        ti0 = time.perf_counter()
        for _ in range(args.steps):
            step(overlap=False)
        torch.cuda.synchronize()
        ms_instr = (time.perf_counter() - ti0) * 1e3 / args.steps
        for c in range(n_cls):
            tot, n = nb.numbat_timing_read(c)
            if n:
                per_cls[nb.numbat_kernel_class_name(c)] = (tot / args.steps, n // args.steps)
        nb.numbat_timing_enable(False)

    pass_flops = sum(l.flops for l in layers)  # one pass (fwd, dgrad or wgrad) over all layers
    roofline = None
    conv_cls = ("conv_fwd_igemm", "conv_dgrad_igemm", "wgrad_igemm")
    if per_cls:
        dom = max((c for c in conv_cls if c in per_cls), key=lambda c: per_cls[c][0])
        dom_ms, dom_launches = per_cls[dom]
        achieved = pass_flops / (dom_ms / 1e3) / 1e12
        traffic = committed_traffic(dom, wl.index, wl.n) if not args.layers else None
        roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic, "kernel": dom,
                    "launches_per_step": dom_launches, "avg_launch_ms": round(dom_ms / max(dom_launches, 1), 4),
                    "flops_per_step": pass_flops}
    conv_ms = sum(per_cls[c][0] for c in per_cls if c not in
                  ("bn_stats", "bn_silu_fwd_apply", "bn_silu_bwd_reduce", "bn_silu_bwd_finalize", "bn_silu_bwd_apply"))
    bn_ms = sum(per_cls[c][0] for c in per_cls) - conv_ms if per_cls else None

    value = step_flops / (ms / 1e3) / 1e12
    out = {
        "metric": "conv fwd+bwd TFLOP/s & % bf16 MFMA peak; ms per YOLOv8m-shape step, batch 16",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name + (f" [{len(layers)} layers]" if args.layers else ""),
                   "config_index": wl.index, "batch": wl.n, "input": "640x640", "layers": len(layers),
                   "mode": "set", "step_gflop": round(step_flops / 1e9, 2),
                   "launch": "hip graph replay" if graph is not None else "eager",
                   "streams": 2 if two else 1,
                   "bn_bwd_in_dgrad_layers": sum(1 for l in layers if l.fused)},
        "pct_mfma_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "roofline": roofline,
        "sclk": sclk.summary(),
    }
    if cold is not None:
        out["ms_per_step_cold_cache"] = cold
    if per_cls:
        out["kernel_ms_per_step"] = {c: round(v[0], 4) for c, v in per_cls.items()}
        out["conv_kernel_ms"] = round(conv_ms, 3)
        out["conv_kernel_tflops"] = round(step_flops / (conv_ms / 1e3) / 1e12, 2)
        out["bn_silu_kernel_ms"] = round(bn_ms, 3)
        out["instrumented_ms_per_step"] = round(ms_instr, 3)
    if args.detail:
        write_detail(torch, args, step, layers, wl)
    copy_gbs = hbm_copy_gbs(torch)
    out["hbm_copy_gbs"] = copy_gbs
    if per_cls:
        # BN + SiLU kernels: algorithmic bytes (bf16) per element of the step's activations --
        # forward apply reads y and writes a (4), backward reduce reads g and y (4), backward
        # apply reads g and y and writes dy (6) -- over their summed kernel time
        # (the backward apply runs only for the layers whose data gradient does not form dy)
        elems = sum(l.bn_elems for l in layers)
        apply_elems = sum(l.bn_elems for l in layers if not l.fused)
        out["bn_silu_gbs"] = {}
        for c, b in (("bn_silu_fwd_apply", 4), ("bn_silu_bwd_reduce", 4), ("bn_silu_bwd_apply", 6)):
            if c in per_cls:
                gbs = b * (apply_elems if c == "bn_silu_bwd_apply" else elems) / (per_cls[c][0] / 1e3) / 1e9
                out["bn_silu_gbs"][c] = {"gbs": round(gbs, 1), "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4),
                                         "frac_copy": round(gbs / copy_gbs, 4)}
    if not args.no_extras and not args.layers and wl.index == 4:
        print("# extras: chain mode, optimiser step, configuration 5", file=sys.stderr, flush=True)
        out["chain_mode"] = chain_mode(torch, args.steps, args.warmup)
        out["optimizer_step"] = optimizer_step(torch, args.steps)
        out["prologue_fusion"] = prologue_fusion(torch, args.steps)
        del graph
        torch.cuda.empty_cache()
        out["config5_batch32"] = config_set(torch, 5, 32, max(5, args.steps // 2), 2)
        out["config5_layers_batch16"] = config_set(torch, 5, 16, max(5, args.steps // 2), 2)
    if not args.no_cpu_baseline:
        print("# cpu baseline (fp64 oracle, bounded sample)", file=sys.stderr, flush=True)
        import oracle

        oracle.build(force=False)
        out["cpu_baseline"] = cpu_baseline(wl, oracle.num_threads())
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
