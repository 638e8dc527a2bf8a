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
    ap.add_argument("--wgrad-group", type=int, default=2,
                    help="deferred order: enqueue the weight gradients in groups of this many layers behind "
                         "one cross-stream wait (each wait costs the main queue a completion signal)")
    ap.add_argument("--wgrad-tail", type=int, default=8,
                    help="the last this many layers of the backward pass are enqueued one by one")
    ap.add_argument("--layers", type=str, default=None, help="comma-separated layer names (subset)")
    ap.add_argument("--detail", type=str, default=None, help="write per-layer timings (JSON) to this file")
    return ap.parse_args()


PASSES = ("conv_fwd", "bn_silu_fwd", "bn_silu_bwd", "conv_bwd_weight", "conv_bwd_data")


# HBM traffic per launch measured with rocprofv3 counters (FETCH_SIZE, WRITE_SIZE, each
# scaled by what it reads for a plain device copy) for a kernel class on one workload; the
# figure is used only while the kernel's sources hash to the value recorded with it.
TRAFFIC_PROFILES = {
    ("wgrad_igemm", 4, 16): ("profiles/wgrad_igemm_c4_b16_traffic.md",
                             ("paper_2609_10632_amd/csrc/conv_wgrad.hip", "paper_2609_10632_amd/csrc/common.h",
                              "paper_2609_10632_amd/csrc/kernels.h")),
    ("conv_fwd_igemm", 4, 16): ("profiles/conv_fwd_igemm_c4_b16_traffic.md",
                                ("paper_2609_10632_amd/csrc/conv_gemm.hip", "paper_2609_10632_amd/csrc/common.h",
                                 "paper_2609_10632_amd/csrc/kernels.h")),
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
                 [wl.layers.index(l) for l in specs])
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
    t0 = time.perf_counter()
    for _ in range(args.steps):
        if graph is not None:
            graph.replay()
        else:
            step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps

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
                   "streams": 2 if two else 1},
        "pct_mfma_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "roofline": roofline,
    }
    if per_cls:
        out["kernel_ms_per_step"] = {c: round(v[0], 4) for c, v in per_cls.items()}
        out["conv_kernel_ms"] = round(conv_ms, 3)
        out["conv_kernel_tflops"] = round(step_flops / (conv_ms / 1e3) / 1e12, 2)
        out["bn_silu_kernel_ms"] = round(bn_ms, 3)
        out["instrumented_ms_per_step"] = round(ms_instr, 3)
    if args.detail:
        ev = {l.name: [torch.cuda.Event(enable_timing=True) for _ in range(7)] for l in layers}
        step(ev, overlap=False)
        torch.cuda.synchronize()
        per_layer = {}
        for l in layers:
            e = ev[l.name]
            per_layer[l.name] = [e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[3].elapsed_time(e[4]),
                                 e[4].elapsed_time(e[5]), e[5].elapsed_time(e[6])]
        with open(args.detail, "w") as f:
            json.dump({"per_layer_ms": per_layer, "passes": PASSES, "flops": {l.name: l.flops for l in layers}}, f,
                      indent=1)
    if not args.no_cpu_baseline:
        print("# cpu baseline (fp64 oracle, bounded sample)", file=sys.stderr, flush=True)
        import oracle

        oracle.build(force=False)
        out["cpu_baseline"] = cpu_baseline(wl, oracle.num_threads())
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
