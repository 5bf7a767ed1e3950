"""Benchmark of the MoCE forward pass on one MI355X.

One step = one ``moce_forward`` over one batch of the workload (pooling,
temperatures, coefficients, routed experts and residual), inputs resident in
HBM.  Consecutive steps rotate over enough distinct (x, y) buffer sets (at
least 1 GiB together) that no step finds its input left in the 256 MB
Infinity Cache by an earlier step.  Timing uses HIP events recorded on the
stream the kernels are launched on.

Prints one JSON line.  ``value`` is the effective bandwidth in GB/s with the
workload's metric bytes (two reads of x, one write of y, the parameters);
``roofline`` prices the dominant kernel's algorithmic bytes against the
8 TB/s HBM peak: the forward runs a pooling kernel and either one kernel for
gate and mix (k = 32 on the MFMA path) or a gate kernel and a mix kernel,
each also reachable through its own entry point; the slowest of them, timed
through that entry point (launches captured in a HIP graph, replays timed
with HIP events), is priced.  ``cpu_baseline``
times the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "MoCE fwd latency (us) + effective HBM GB/s (% of peak) at ResNet-50 shapes"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="resnet50_stage1")
    p.add_argument("--layout", default=None)
    p.add_argument("--rotate-gib", type=float, default=1.0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--no-context", action="store_true")
    # after the measurements, copy this many MiB device to device five times:
    # a plain copy kernel of known size against which hardware byte counters
    # (rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE) are calibrated
    p.add_argument("--copy-probe-mib", type=int, default=0)
    return p.parse_args()


def measured_traffic(kernel: str):
    """HBM-side bytes per launch of `kernel` from the committed rocprofv3 byte
    counters (calibrated against a plain copy), or None when the kernel's
    sources have changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "mix_resnet50_stage1_hbm_bytes.md")
    if not os.path.exists(path):
        return None
    rec = {}
    for ln in open(path):
        k, sep, v = ln.partition(":")
        if sep and k.strip() in ("kernel", "sources", "sources_sha256", "traffic_bytes"):
            rec[k.strip()] = v.strip()
    if rec.get("kernel") != kernel or "sources" not in rec:
        return None
    h = hashlib.sha256()
    for f in rec["sources"].split():
        fp = os.path.join(ROOT, f)
        if not os.path.exists(fp):
            return None
        h.update(open(fp, "rb").read())
    if h.hexdigest() != rec.get("sources_sha256"):
        return None
    return int(rec["traffic_bytes"])


def launch_time_ms(fn, n, reps=3):
    """Average duration of one launch of fn(i): the launches of fn(0) ..
    fn(n-1) are captured in one HIP graph (so no host time falls between
    them) and the graph's replays are timed with HIP events on the stream
    that replays it; best of `reps` replays."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(min(n, 3)):
            fn(i, side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        st = torch.cuda.current_stream()
        for i in range(n):
            fn(i, st)
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    best = None
    for _ in range(reps):
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        st = torch.cuda.current_stream()
        t0.record(st)
        graph.replay()
        t1.record(st)
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / n
        best = ms if best is None else min(best, ms)
    return best


def event_time_ms(fn, n, stream):
    import torch
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(n):
        fn(i)
    t1.record(stream)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / n


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(images are independent, so a batch-sharded run needs no communication and scales "
              "with the per-GPU share).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_23794_amd import binding as mb
    from paper_2608_23794_amd import cost, inputs
    from paper_2608_23794_amd.layer import MoceLayer, to_device_x

    wl = inputs.WORKLOADS[args.workload]
    layout = args.layout or wl.layouts[0]
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    g = inputs.generate(wl, layout)
    layer = MoceLayer.from_workload(wl, g, layout)
    if layer.status != 0:
        raise RuntimeError(f"support preparation failed: status {layer.status}")
    B = wl.B
    traffic = cost.layer_traffic(B, wl.C, wl.E, wl.k, wl.HW, wl.elem_bytes)
    per_set = traffic["x"] + traffic["y"]
    nsets = max(1, math.ceil(args.rotate_gib * 2 ** 30 / per_set))
    x0 = to_device_x(g["x"], wl.dtype)
    xs = [x0] + [x0.clone() for _ in range(nsets - 1)]
    ys = [torch.empty(layer.y_shape(B), dtype=x0.dtype, device="cuda") for _ in range(nsets)]
    ws = layer.new_workspace(B)

    def step(i):
        layer.forward(xs[i % nsets], ys[i % nsets], ws)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms = event_time_ms(step, args.steps, stream)
    ms_warm = event_time_ms(lambda i: layer.forward(xs[0], ys[0], ws), max(args.steps // 2, 1), stream)

    # per-kernel times of the same work through the stage entry points (the
    # inputs rotate as in the forward's timing, so the mix reads x that is not
    # in the infinity cache, unlike the forward's mix)
    d = torch.empty((B, wl.C), dtype=torch.float32, device="cuda")
    tau = torch.empty((B, wl.E - 1), dtype=torch.float32, device="cuda")
    alpha = torch.empty((B, wl.E - 1, wl.k), dtype=torch.float32, device="cuda")
    desc = layer.desc(B)
    n_k = max(args.steps // 2, 10)
    U = layer.U if layer.nU else None
    t_pool = launch_time_ms(lambda i, st: mb.moce_pool(desc, xs[i % nsets], d, st), n_k)
    t_gate = launch_time_ms(lambda i, st: mb.moce_gate(desc, d, layer.s_c, layer.w_c, layer.gate, tau, alpha, st),
                            n_k)
    t_mix = launch_time_ms(lambda i, st: mb.moce_mix(desc, xs[i % nsets], layer.s_c, alpha, U, layer.nU,
                                                     ys[i % nsets], st), n_k)
    R, k = wl.E - 1, wl.k
    stages = {
        "pool": (t_pool, traffic["x"] + B * wl.C * 4),
        "gate": (t_gate, B * R * k * 4 + R * k * 12 + B * R * 4 + B * R * k * 4),
        "mix": (t_mix, traffic["x"] + traffic["y"] + B * R * k * 4 + R * k * 4),
    }
    path = mb.moce_forward_path(desc, mb.MOCE_GATE_SOFTPLUS_LINEAR)
    if path == mb.PATH_MFMA_GATE:
        # the forward's second kernel: gate and mix in one (x, y, the pooled
        # descriptors, supports, slopes, logits and offsets)
        t_gm = launch_time_ms(lambda i, st: mb.moce_gate_mix(desc, xs[i % nsets], d, layer.s_c, layer.w_c,
                                                             layer.gate, U, layer.nU, ys[i % nsets], st), n_k)
        kernels = {"pool": stages["pool"],
                   "gate_mix": (t_gm, traffic["x"] + traffic["y"] + B * wl.C * 4 + R * k * 12 + R * 4)}
    else:
        kernels = stages
    dom = max(kernels, key=lambda n: kernels[n][0])
    dom_ms, dom_bytes = kernels[dom]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9

    value = traffic["metric"] / (ms * 1e-3) / 1e9
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "accumulate": "f32",
        "data": "synthetic (seeded, shapes and distributions of the named layer)",
        "config": {**wl.describe(), "layout": layout,
                   "forward": {mb.PATH_TILE: "pool, gate, tile mix",
                               mb.PATH_MFMA_GATE: "pool, gate inside the mix"}.get(path, "pool, gate, mix")},
        "latency_us": round(ms * 1e3, 2),
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 1),
        "latency_us_warm_cache": round(ms_warm * 1e3, 2),
        "bytes": {"metric": traffic["metric"], "compulsory": traffic["compulsory"]},
        "compulsory_GBps": round(traffic["compulsory"] / (ms * 1e-3) / 1e9, 1),
        "rotation_sets": nsets,
        "kernels_us": {n: round(v[0] * 1e3, 2) for n, v in kernels.items()},
        "stage_entry_points_us": {n: round(v[0] * 1e3, 2) for n, v in stages.items()},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(f"k_mfmamix<{wl.C // 32}, 3, {'true' if dom == 'gate_mix' else 'false'}>")
                     if dom in ("mix", "gate_mix") and path in (mb.PATH_MFMA, mb.PATH_MFMA_GATE) else None,
                     "algorithmic_bytes": dom_bytes},
    }

    if not args.no_context:
        C, E = wl.C, wl.E
        Wd = torch.randn((E, C), device="cuda", dtype=torch.float32).to(x0.dtype)
        if layout == "nchw":
            W4 = Wd.view(E, C, 1, 1)
            dense = lambda i: torch.nn.functional.conv2d(xs[i % nsets], W4)
        else:
            dense = lambda i: xs[i % nsets].view(-1, C) @ Wd.t()
        for i in range(5):
            dense(i)
        t_dense = event_time_ms(dense, max(args.steps // 2, 10), stream)
        line["context"] = {"dense_1x1_us": round(t_dense * 1e3, 2),
                           "dense_1x1_GBps_x_plus_y": round(per_set / (t_dense * 1e-3) / 1e9, 1),
                           "moce_over_dense_time": round(ms / t_dense, 3)}

    if not args.no_cpu_baseline:
        import oracle
        oracle.build(force=False)
        ol = oracle.NCHW if layout == "nchw" else oracle.NHWC
        s_c, w_c, _, U_h, _ = oracle.prepare(wl.C, wl.E, g["s"], g["w"])
        passes, t_start = 0, time.perf_counter()
        while True:
            dd = oracle.pool(g["x"], ol)
            tt = oracle.gate_softplus(dd, s_c, g["a"], g["c"])
            al = oracle.softmax(w_c, tt)
            oracle.mix(g["x"], s_c, al, U_h, wl.E, ol)
            passes += 1
            if time.perf_counter() - t_start >= args.cpu_seconds:
                break
        per_pass = (time.perf_counter() - t_start) / passes
        line["cpu_baseline"] = {"value": round(traffic["metric"] / per_pass / 1e9, 3), "unit": "GB/s",
                                "cores": oracle.threads(), "kind": "oracle",
                                "sample": f"{passes} full-batch forward passes of {wl.name} (B={B}), "
                                          f"{per_pass * 1e3:.1f} ms each, os.cpu_count()={os.cpu_count()}"}
    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib * 2 ** 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
