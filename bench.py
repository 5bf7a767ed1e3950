"""Benchmark of the MoCE forward pass on one MI355X.

One step = one ``moce_forward`` over one batch of the workload (pooling,
temperatures, coefficients, routed experts and residual), inputs resident in
HBM.  Consecutive steps rotate over enough distinct (x, y) buffer sets (at
least 1 GiB together) that no step finds its input left in the 256 MB
Infinity Cache by an earlier step.  Timing uses HIP events recorded on the
stream the kernels are launched on.

Prints one JSON line for the headline workload (ResNet-50 stage-1 by
default).  ``value`` is the effective bandwidth in GB/s with the workload's
metric bytes (two reads of x, one write of y, the parameters) over the mean
step time of the K timed steps; ``latency_us_median`` / ``latency_us_iqr``
come from a second run of K steps with an event recorded between every two.  ``roofline`` prices the
dominant kernel's algorithmic bytes against the 8 TB/s HBM peak: each kernel
the forward runs is timed through its own entry point (launches captured in a
HIP graph, replays timed with HIP events).  ``other_configs`` repeats the
measurement for the other workloads (stage 3 in both layouts, stage 4, the ViT
token layer), with forwards captured in HIP graphs so that host time never
enters.  ``cpu_baseline`` times the CPU oracle on a bounded sample of the
headline workload, with all host threads and with one.
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
OTHER = (("resnet50_stage3", "nchw"), ("resnet50_stage3", "nhwc"), ("resnet50_stage4", "nhwc"),
         ("vit_tokens", "nhwc"))


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
    p.add_argument("--no-other", action="store_true", help="skip the other workloads")
    p.add_argument("--no-replaced-ops", action="store_true", help="skip the ResNet-50 replaced-operator timing")
    p.add_argument("--gate", default="softplus", choices=("softplus", "mlp"),
                   help="gate kind of the headline workload (the benchmark configurations use softplus)")
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


def _capture(fn, n):
    """A HIP graph of the launches fn(0, st) .. fn(n-1, st), after a few eager
    warm-up calls on a side stream."""
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
    return graph


def graph_times_ms(fn, n, reps):
    """Per-launch duration of fn, once per replay: the launches of fn(0) ..
    fn(n-1) are captured in one HIP graph (so no host time falls between
    them) and each of `reps` replays is timed with HIP events on the stream
    that replays it."""
    import torch
    graph = _capture(fn, n)
    out = []
    for _ in range(reps):
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        st = torch.cuda.current_stream()
        t0.record(st)
        graph.replay()
        t1.record(st)
        torch.cuda.synchronize()
        out.append(t0.elapsed_time(t1) / n)
    return out


def launch_time_ms(fn, n, reps=3):
    """Best per-launch duration over `reps` graph replays (see graph_times_ms)."""
    return min(graph_times_ms(fn, n, reps))


def timed_steps(fn, n, stream):
    """Runs fn(0) .. fn(n-1) eagerly between two synchronisations, with an
    event recorded on `stream` before each step and after the last.  Returns
    (mean ms per step over the bracketed region, per-step ms list)."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    torch.cuda.synchronize()
    for i in range(n):
        ev[i].record(stream)
        fn(i)
    ev[n].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(n)]
    return ev[0].elapsed_time(ev[n]) / n, per


def mean_steps(fn, n, stream):
    """Mean ms per step of fn(0) .. fn(n-1), run eagerly between two
    synchronisations with one event before the first and one after the last."""
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


def quartiles(v):
    import numpy as np
    q1, q2, q3 = np.percentile(np.asarray(v, dtype=np.float64), [25, 50, 75])
    return float(q1), float(q2), float(q3)


class Bench:
    """Device inputs and timers for one workload and layout."""

    def __init__(self, name, layout, rotate_gib, gate="softplus"):
        import torch

        from paper_2608_23794_amd import binding as mb
        from paper_2608_23794_amd import cost, inputs
        from paper_2608_23794_amd.layer import MoceLayer, to_device_x

        self.mb = mb
        self.wl = wl = inputs.WORKLOADS[name]
        self.layout = layout or wl.layouts[0]
        self.g = g = inputs.generate(wl, self.layout)
        self.layer = layer = MoceLayer.from_workload(wl, g, self.layout, gate=gate)
        self.gate_kind = mb.MOCE_GATE_SOFTPLUS_LINEAR if gate == "softplus" else mb.MOCE_GATE_MLP_SIGMOID
        self.B = B = wl.B
        self.traffic = cost.layer_traffic(B, wl.C, wl.E, wl.k, wl.HW, wl.elem_bytes)
        per_set = self.traffic["x"] + self.traffic["y"]
        self.per_set = per_set
        self.nsets = nsets = max(1, math.ceil(rotate_gib * 2 ** 30 / per_set))
        x0 = to_device_x(g["x"], wl.dtype)
        self.xs = [x0] + [x0.clone() for _ in range(nsets - 1)]
        self.ys = [torch.empty(layer.y_shape(B), dtype=x0.dtype, device="cuda") for _ in range(nsets)]
        self.ws = layer.new_workspace(B)
        self.desc = layer.desc(B)
        self.U = layer.U if layer.nU else None
        self.path = mb.moce_forward_path(self.desc, self.gate_kind)
        del g["x"]

    def forward(self, i, st=None):
        n = i % self.nsets
        self.layer.forward(self.xs[n], self.ys[n], self.ws)

    def stage_times(self, n_k):
        """Each kernel of the forward timed through its own entry point (HIP
        graph replays), with its algorithmic bytes."""
        import torch
        mb, wl, B, L = self.mb, self.wl, self.B, self.layer
        R, k, C = wl.E - 1, wl.k, wl.C
        d = torch.empty((B, C), dtype=torch.float32, device="cuda")
        tau = torch.empty((B, R), dtype=torch.float32, device="cuda")
        alpha = torch.empty((B, R, k), dtype=torch.float32, device="cuda")
        desc, nsets, xs, ys, U = self.desc, self.nsets, self.xs, self.ys, self.U
        t_pool = launch_time_ms(lambda i, st: mb.moce_pool(desc, xs[i % nsets], d, st), n_k)
        t_gate = launch_time_ms(lambda i, st: mb.moce_gate(desc, d, L.s_c, L.w_c, L.gate, tau, alpha, st), n_k)
        t_mix = launch_time_ms(lambda i, st: mb.moce_mix(desc, xs[i % nsets], L.s_c, alpha, U, L.nU,
                                                         ys[i % nsets], st), n_k)
        tr = self.traffic
        stages = {
            "pool": (t_pool, tr["x"] + B * C * 4),
            "gate": (t_gate, B * R * k * 4 + R * k * 12 + B * R * 4 + B * R * k * 4),
            "mix": (t_mix, tr["x"] + tr["y"] + B * R * k * 4 + R * k * 4),
        }
        if self.path == mb.PATH_MFMA_GATE:
            t_gm = launch_time_ms(lambda i, st: mb.moce_gate_mix(desc, xs[i % nsets], d, L.s_c, L.w_c, L.gate, U,
                                                                 L.nU, ys[i % nsets], st), n_k)
            kernels = {"pool": stages["pool"],
                       "gate_mix": (t_gm, tr["x"] + tr["y"] + B * C * 4 + R * k * 12 + R * 4)}
        elif self.path == mb.PATH_SCHEDULED:
            # no entry point runs the scheduled mix alone: its time is the
            # forward's less the pool and gate entry points (the schedule
            # build, beside the pooling or after it, is counted with the mix)
            t_fwd = launch_time_ms(lambda i, st: self.forward(i, st), n_k)
            kernels = {"pool": stages["pool"], "gate": stages["gate"],
                       "scheduled_mix": (max(t_fwd - t_pool - t_gate, 1e-6),
                                         tr["x"] + tr["y"] + 3 * B * R * 4)}
        else:
            kernels = stages
        return stages, kernels

    def dense_context(self, n, stream):
        import torch
        wl, nsets, xs = self.wl, self.nsets, self.xs
        C, E = wl.C, wl.E
        Wd = torch.randn((E, C), device="cuda", dtype=torch.float32).to(xs[0].dtype)
        if self.layout == "nchw":
            W4 = Wd.view(E, C, 1, 1)
            dense = lambda i: torch.nn.functional.conv2d(xs[i % nsets], W4)
        else:
            dense = lambda i: xs[i % nsets].view(-1, C) @ Wd.t()
        for i in range(5):
            dense(i)
        t = mean_steps(dense, n, stream)
        return {"dense_1x1_us": round(t * 1e3, 2),
                "dense_1x1_GBps_x_plus_y": round(self.per_set / (t * 1e-3) / 1e9, 1)}

    def release(self):
        import torch
        self.xs = self.ys = None
        torch.cuda.empty_cache()


def roofline_entry(kernels, path, mb, C):
    dom = max(kernels, key=lambda n: kernels[n][0])
    dom_ms, dom_bytes = kernels[dom]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    traffic = None
    if dom in ("mix", "gate_mix") and path in (mb.PATH_MFMA, mb.PATH_MFMA_GATE):
        traffic = measured_traffic(f"k_mfmamix<{C // 32}, 3, {'true' if dom == 'gate_mix' else 'false'}>")
    return {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic, "algorithmic_bytes": dom_bytes}


FORWARD_NAMES = {0: "pool, gate, mix", 1: "pool, gate, tile mix", 2: "pool, gate, matrix-core mix",
                 3: "pool, gate inside the matrix-core mix",
                 4: "pool with the support schedule, gate statistics, scheduled matrix-core mix",
                 5: "pool, gate, channels-last gather"}

# workloads whose line carries both gate forms timed through the gate entry point
GATE_TIMED = ("resnet50_stage1", "resnet50_stage4")


def gate_forms_us(bn, n_k):
    """moce_gate of this workload with the softplus-linear gate and with the
    paper's MLP gate (batched product), temperatures only, on the pooled
    descriptor of the first input set."""
    import torch
    from paper_2608_23794_amd.layer import MoceLayer
    mb, wl, B = bn.mb, bn.wl, bn.B
    R, C = wl.E - 1, wl.C
    d = torch.empty((B, C), dtype=torch.float32, device="cuda")
    mb.moce_pool(bn.desc, bn.xs[0], d, torch.cuda.current_stream())
    tau = torch.empty((B, R), dtype=torch.float32, device="cuda")
    out = {}
    for form in ("softplus", "mlp"):
        L = bn.layer if form == "softplus" else MoceLayer.from_workload(wl, bn.g, bn.layout, gate="mlp")
        t = launch_time_ms(lambda i, st: mb.moce_gate(bn.desc, d, L.s_c, L.w_c, L.gate, tau, None, st), n_k)
        out[form] = round(t * 1e3, 2)
    return out


def dynamic_us(bn, n_g=10, reps=5):
    """The input-conditioned variant (router width 32, synthetic router of the workload's
    shape) timed like the static forward: HIP graph of n_g forwards, median of reps replays."""
    import torch
    from paper_2608_23794_amd import inputs
    from paper_2608_23794_amd.layer import DynamicMoceLayer
    dl = DynamicMoceLayer.from_workload(bn.wl, bn.g, inputs.router_params(bn.wl), bn.layout)
    ws = dl.new_workspace(bn.B)
    t = quartiles(graph_times_ms(lambda i, st=None: dl.forward(bn.xs[i % bn.nsets], bn.ys[i % bn.nsets], ws), n_g, reps))[1]
    del ws
    torch.cuda.empty_cache()
    return t


def backward_us(bn, n_g=5, reps=5):
    """moce_backward (dx, dw and the gate's gradients for a random upstream dy) timed like the
    forward: HIP graph of n_g calls over the rotating input sets, median of reps replays.
    Returns (latency in ms, compulsory bytes: x and dy read once, dx written once)."""
    import torch
    layer = bn.layer
    x0 = bn.xs[0]
    dy = torch.randn(layer.y_shape(bn.B), device="cuda").to(x0.dtype)
    dx = torch.empty_like(x0)
    ws = layer.new_backward_workspace(bn.B)
    t = quartiles(graph_times_ms(lambda i, st=None: layer.backward(bn.xs[i % bn.nsets], dy, dx, ws), n_g, reps))[1]
    nbytes = 2 * x0.numel() * x0.element_size() + dy.numel() * dy.element_size()
    del ws, dx, dy
    torch.cuda.empty_cache()
    return t, nbytes


def epilogue_entry(bn, fwd_ms, n_g=10, reps=5):
    """The forward with the fused output epilogue (per-channel affine map and ReLU: a folded inference
    batch norm), against the plain forward and against the same epilogue as a separate torch pass over
    y (y * scale + shift, then ReLU), all as HIP-graph replays."""
    import torch
    E = bn.wl.E
    scale = (torch.rand(E, device="cuda") + 0.5).float()
    shift = (torch.randn(E, device="cuda") * 0.1).float()
    ep = (scale, shift, True)
    t_fused = quartiles(graph_times_ms(
        lambda i, st=None: bn.layer.forward(bn.xs[i % bn.nsets], bn.ys[i % bn.nsets], bn.ws, epilogue=ep), n_g, reps))[1]
    shp = [1, E, 1, 1] if bn.layout == "nchw" else [1, 1, 1, E]
    sc, sf = scale.view(shp).to(bn.ys[0].dtype), shift.view(shp).to(bn.ys[0].dtype)

    def separate(i, st=None):
        y = bn.ys[i % bn.nsets]
        bn.layer.forward(bn.xs[i % bn.nsets], y, bn.ws)
        torch.relu_(y.mul_(sc).add_(sf))
    t_sep = quartiles(graph_times_ms(separate, n_g, reps))[1]
    return {"fused_us": round(t_fused * 1e3, 2), "plain_forward_us": round(fwd_ms * 1e3, 2),
            "forward_then_torch_pass_us": round(t_sep * 1e3, 2),
            "timing": "HIP graph of 10 forwards, median of 5 replays; epilogue = ReLU(scale * y + shift) per output channel"}


def backward_entry(bn, fwd_ms):
    t, nbytes = backward_us(bn)
    return {"latency_us": round(t * 1e3, 2), "compulsory_bytes": nbytes, "GBps": round(nbytes / (t * 1e-3) / 1e9, 1),
            "over_forward": round(t / fwd_ms, 2),
            "timing": "HIP graph of 5 calls, median of 5 replays; dx, dw and the softplus-linear gate's gradients"}


# The entrance 1x1 projections of the ResNet-50 bottleneck blocks, which the paper replaces (Sec. 4.1):
# (input channels, outputs, spatial size, blocks)
RESNET50_ENTRANCES = ((64, 64, 56, 1), (256, 64, 56, 2), (256, 128, 56, 1), (512, 128, 28, 3),
                      (512, 256, 28, 1), (1024, 256, 14, 5), (1024, 512, 14, 1), (2048, 512, 7, 2))


def replaced_ops(batch=512, k=8, n_g=3, reps=5):
    """Every replaced operator of ResNet-50 (the 16 entrance projections) as MoCE layers with random
    weights and supports (k = 8, the paper's ResNet setting), timed against the dense 1x1 projection
    at the same shape: both channels-last bf16, batch 512, HIP graphs of n_g calls, median of reps
    replays.  The dense projection is one GEMM [B H W, C] x [C, E] through torch (hipBLASLt)."""
    import numpy as np
    import torch
    from paper_2608_23794_amd import binding as mb
    from paper_2608_23794_amd.layer import MoceLayer
    rng = np.random.default_rng(2608)
    rows, t_moce, t_dense = [], 0.0, 0.0
    for C, E, S, nblk in RESNET50_ENTRANCES:
        R = E - 1
        s = np.array([rng.choice(C, size=k, replace=False) for _ in range(R)], np.int32)
        w = rng.standard_normal((R, k)).astype(np.float32)
        a = (rng.standard_normal((R, k)) / np.sqrt(k)).astype(np.float32)
        layer = MoceLayer(C, E, k, S, S, "bf16", "nhwc", s, w, a=a, c=np.zeros(R, np.float32))
        x = torch.relu(torch.randn((batch, S, S, C), device="cuda")).to(torch.bfloat16)
        y = torch.empty(layer.y_shape(batch), dtype=torch.bfloat16, device="cuda")
        ws = layer.new_workspace(batch)
        tm = quartiles(graph_times_ms(lambda i, st=None: layer.forward(x, y, ws), n_g, reps))[1]
        Wd = (torch.randn((C, E), device="cuda") / math.sqrt(C)).to(torch.bfloat16)
        x2 = x.view(-1, C)
        yd = torch.empty((x2.shape[0], E), dtype=torch.bfloat16, device="cuda")
        td = quartiles(graph_times_ms(lambda i, st=None: torch.matmul(x2, Wd, out=yd), n_g, reps))[1]
        path = mb.moce_forward_path(layer.desc(batch), mb.MOCE_GATE_SOFTPLUS_LINEAR)
        rows.append({"shape": f"{C}->{E} @{S}x{S}", "blocks": nblk, "forward": FORWARD_NAMES.get(path, str(path)),
                     "moce_us": round(tm * 1e3, 1),
                     "dense_us": round(td * 1e3, 1), "moce_over_dense": round(tm / td, 3)})
        t_moce += nblk * tm
        t_dense += nblk * td
        del x, y, ws, x2, yd, Wd, layer, path
        torch.cuda.empty_cache()
    return {"network": "ResNet-50, the 16 bottleneck entrance projections", "batch": batch, "k": k,
            "dtype": "bf16", "layout": "channels-last", "weights": "random",
            "moce_total_ms": round(t_moce, 3), "dense_total_ms": round(t_dense, 3),
            "moce_over_dense": round(t_moce / t_dense, 3), "per_shape": rows,
            "paper_context": "float32, batch 512, the paper's GPU: 15.60 ms against 19.63 ms for all replaced "
                             "operators; the 2048->512 module at 0.331 of the dense time (Sec. 4.7, Table 7)"}


def other_config(name, layout, args, stream):
    bn = Bench(name, layout, args.rotate_gib)
    mb, wl = bn.mb, bn.wl
    n_g = 20
    reps = 15
    fwd = graph_times_ms(bn.forward, n_g, reps)
    q1, med, q3 = quartiles(fwd)
    stages, kernels = bn.stage_times(n_g)
    rf = roofline_entry(kernels, bn.path, mb, wl.C)
    out = {
        "workload": name, "layout": layout, "B": wl.B, "C_in": wl.C, "C_out": wl.E, "k": wl.k,
        "H": wl.H, "W": wl.W, "dtype": wl.dtype, "forward": FORWARD_NAMES.get(bn.path, str(bn.path)),
        "latency_us": round(med * 1e3, 2), "latency_us_iqr": [round(q1 * 1e3, 2), round(q3 * 1e3, 2)],
        "timing": f"HIP graph of {n_g} forwards over {bn.nsets} rotating input sets, median of {reps} replays",
        "GBps": round(bn.traffic["metric"] / (med * 1e-3) / 1e9, 1),
        "pct_of_hbm_peak": round(100 * bn.traffic["metric"] / (med * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
        "stage_entry_points_us": {n: round(v[0] * 1e3, 2) for n, v in stages.items()},
        "dominant_kernel": rf["kernel"], "dominant_kernel_us": round(kernels[rf["kernel"]][0] * 1e3, 2),
        "roofline_frac": rf["frac"],
    }
    if bn.path == mb.PATH_SCHEDULED:
        out["stage_entry_points_note"] = ("the entry points time the generic pool, gate and coefficient mix; the "
                                          "scheduled mix is timed as the forward less the pool and gate entry "
                                          "points, and per kernel in its rocprofv3 summaries")
    if name in GATE_TIMED:
        out["gate_entry_point_us"] = gate_forms_us(bn, n_g)
    t_dyn = dynamic_us(bn)
    out["dynamic_supports"] = {"latency_us": round(t_dyn * 1e3, 2), "over_static": round(t_dyn / med, 2),
                               "router_width": 32}
    out["backward"] = backward_entry(bn, med)
    out["bn_relu_epilogue"] = epilogue_entry(bn, med)
    if not args.no_context:
        out["context"] = bn.dense_context(max(args.steps // 4, 10), stream)
        out["context"]["moce_over_dense_time"] = round(med * 1e3 / out["context"]["dense_1x1_us"], 3)
    bn.release()
    return out


def cpu_baseline(bench, seconds):
    import oracle
    oracle.build(force=False)
    wl, g, layout = bench.wl, bench.g, bench.layout
    from paper_2608_23794_amd import inputs
    x = inputs.generate(wl, layout)["x"]
    ol = oracle.NCHW if layout == "nchw" else oracle.NHWC
    s_c, w_c, _, U_h, _ = oracle.prepare(wl.C, wl.E, g["s"], g["w"])

    def one_pass():
        dd = oracle.pool(x, ol)
        tt = oracle.gate_softplus(dd, s_c, g["a"], g["c"])
        al = oracle.softmax(w_c, tt)
        oracle.mix(x, s_c, al, U_h, wl.E, ol)

    def run(limit):
        passes, t_start = 0, time.perf_counter()
        while True:
            one_pass()
            passes += 1
            if time.perf_counter() - t_start >= limit:
                break
        return passes, (time.perf_counter() - t_start) / passes

    all_threads = oracle.threads()
    passes, per_pass = run(seconds)
    oracle.set_threads(1)
    p1, per_pass_1 = run(max(seconds / 3, 1.0))
    oracle.set_threads(all_threads)
    metric = bench.traffic["metric"]
    return {"value": round(metric / per_pass / 1e9, 3), "unit": "GB/s", "cores": all_threads, "kind": "oracle",
            "sample": f"{passes} full-batch forward passes of {wl.name} (B={wl.B}), {per_pass * 1e3:.1f} ms each "
                      f"on {all_threads} threads",
            "single_thread": {"value": round(metric / per_pass_1 / 1e9, 4), "unit": "GB/s",
                              "ms_per_pass": round(per_pass_1 * 1e3, 1), "passes": p1},
            "os_cpu_count": os.cpu_count(), "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(images are independent, so a batch-sharded run needs no communication and scales "
              "with the per-GPU share).", file=sys.stderr)
        sys.exit(2)

    import torch

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    bn = Bench(args.workload, args.layout, args.rotate_gib, gate=args.gate)
    mb, wl = bn.mb, bn.wl
    if bn.layer.status != 0:
        raise RuntimeError(f"support preparation failed: status {bn.layer.status}")

    for i in range(args.warmup):
        bn.forward(i)
    torch.cuda.synchronize()
    # the K timed steps with events only around them (the headline), then the
    # same number of steps with an event between every two (the per-step
    # distribution; an event between kernels can add a gap of its own)
    ms = mean_steps(bn.forward, args.steps, stream)
    _, per = timed_steps(bn.forward, args.steps, stream)
    q1, med, q3 = quartiles(per)
    ms_warm = mean_steps(lambda i: bn.layer.forward(bn.xs[0], bn.ys[0], bn.ws), max(args.steps // 2, 1), stream)
    fwd_graph = quartiles(graph_times_ms(bn.forward, 20, 15))[1]

    stages, kernels = bn.stage_times(max(args.steps // 2, 10))
    roof = roofline_entry(kernels, bn.path, mb, wl.C)
    value = bn.traffic["metric"] / (ms * 1e-3) / 1e9
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
        "config": {**wl.describe(), "layout": bn.layout, "gate": args.gate,
                   "forward": FORWARD_NAMES.get(bn.path, str(bn.path))},
        "latency_us": round(ms * 1e3, 2),
        "latency_us_median": round(med * 1e3, 2),
        "latency_us_iqr": [round(q1 * 1e3, 2), round(q3 * 1e3, 2)],
        "latency_us_graph": round(fwd_graph * 1e3, 2),
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 1),
        "latency_us_warm_cache": round(ms_warm * 1e3, 2),
        "bytes": {"metric": bn.traffic["metric"], "compulsory": bn.traffic["compulsory"]},
        "compulsory_GBps": round(bn.traffic["compulsory"] / (ms * 1e-3) / 1e9, 1),
        "rotation_sets": bn.nsets,
        "kernels_us": {n: round(v[0] * 1e3, 2) for n, v in kernels.items()},
        "stage_entry_points_us": {n: round(v[0] * 1e3, 2) for n, v in stages.items()},
        "roofline": roof,
    }
    if wl.name in GATE_TIMED:
        line["gate_entry_point_us"] = gate_forms_us(bn, max(args.steps // 2, 10))
    t_dyn = dynamic_us(bn)
    line["dynamic_supports"] = {"latency_us": round(t_dyn * 1e3, 2), "over_static": round(t_dyn / fwd_graph, 2),
                                "router_width": 32,
                                "timing": "HIP graph of 10 forwards, median of 5 replays; over the static graph latency"}
    line["backward"] = backward_entry(bn, fwd_graph)
    line["bn_relu_epilogue"] = epilogue_entry(bn, fwd_graph)
    if not args.no_context:
        line["context"] = bn.dense_context(max(args.steps // 2, 10), stream)
        line["context"]["moce_over_dense_time"] = round(ms * 1e3 / line["context"]["dense_1x1_us"], 3)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(bn, args.cpu_seconds)
    bn.release()

    if not args.no_other:
        others = {}
        for name, layout in OTHER:
            if (name, layout) == (args.workload, bn.layout):
                continue
            print(f"# bench: {name}/{layout}", file=sys.stderr, flush=True)
            others[f"{name}/{layout}"] = other_config(name, layout, args, stream)
        line["other_configs"] = others

    if not args.no_replaced_ops:
        print("# bench: replaced operators", file=sys.stderr, flush=True)
        line["replaced_ops"] = replaced_ops()

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
