#!/usr/bin/env python3
"""Benchmark: fp32 convolution training passes on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
the forward pass of every layer of a conv stack, then, in reverse layer
order, the backward-weight (+ bias) and backward-data passes (the network's
first layer skips backward-data, whose result no layer would use).  Every
layer occurs as many times as the stack lists it.

Default workload: the VGG-16-shaped stack, batch 32, input 3x224x224 (the
largest configuration; the network behind the paper's per-pass Table II).
Printed: ONE JSON line with images/s of the stack (value), TFLOP/s per pass
(2 N K P Q (C/G) R S flops per pass, divided by the device time of the
whole library call), the roofline fraction of the dominant kernel, the
measured reference points of the chip (fp32 matrix-core loop, HBM copy,
shader clock), and the CPU oracle timed on a bounded sample of the same
workload.

All inputs are resident in device memory before the timed region; the timed
region contains only the library's calls.  Two schedules of the step exist:
every pass on torch's current stream, or each layer's backward-weight pass
on a second stream beside its backward-data pass, ordered by events as the
data dependencies of a training step require (a layer's dy exists once the
backward-data pass of the layer above it has run).  By default (--streams 0)
both are timed over a few steps after the warm-up and the faster one is
used (the event hand-offs cost more than they gain on launch-bound stacks);
--streams 1 or 2 forces one.  Per-pass figures and the dominant kernel are
timed alone on the current stream, from warm caches; passes whose HBM
bytes weigh at least half as much as their flops in the roofline are also
timed from cold caches (a 512 MiB buffer written between repeats).  Before
the warm-up, every layer pass is tuned (conv_tune: each candidate plan is
timed on the layer's tensors and the fastest kept, as the paper's framework
picks its convolution strategy over the first training iterations);
--tune 0 keeps the library's built-in rule instead.  With --graph 1 the step
is captured once into a HIP graph (on a side stream) and its replays are
timed instead of eager calls.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fp32 conv TFLOP/s per pass (fwd/bwdD/bwdW) + images/s conv stack"
PEAK_TFLOPS = 157.3   # MI355X dense fp32 MFMA
PEAK_GBS = 8000.0     # MI355X HBM3E
PASSES = ("fwd", "bwd_data", "bwd_weight")

WORKLOAD_NAMES = {
    0: "single conv layer N=2 C=16 32x32 K=32 3x3 s1 p1 (all three passes)",
    1: "AlexNet-shaped conv stack fwd+bwd, batch 128, input 3x227x227 (5 conv layers)",
    2: "VGG-16-shaped conv stack fwd+bwd, batch 32, input 3x224x224 (13 conv layers)",
    3: "ResNet-50-shaped bottleneck conv set fwd+bwd, batch 64 (stem, 4 stages, projections)",
    4: "GoogLeNet-inception-shaped conv set fwd+bwd, batch 64 (3 modules on 28x28/14x14)",
    5: "AlexNet-shaped network step fwd+bwd, batch 128: 5 conv, 3 max-pool (3x3/2), "
       "3 inner-product layers (no element-wise layers)",
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="2", help="0-5, or 'all' (one JSON line each)")
    ap.add_argument("--reps", type=int, default=20, help="timed repeats per layer and pass")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample (0 disables it)")
    ap.add_argument("--tune", type=int, default=3, metavar="REPS",
                    help="before the warm-up, time every candidate plan of every layer pass "
                         "with REPS runs and keep the fastest (0: the built-in rule)")
    ap.add_argument("--flush", action="store_true",
                    help="time every per-layer pass from cold caches too (a 512 MiB buffer "
                         "written between repeats), not only the memory-bound ones")
    ap.add_argument("--profile-pass", default=None, metavar="CFG:LAYER:PASS",
                    help="only run one layer pass --reps times (for rocprofv3), print nothing else")
    ap.add_argument("--plan", type=int, default=None, metavar="INDEX",
                    help="with --profile-pass: run candidate plan INDEX (conv_plan_set) "
                         "instead of tuning")
    ap.add_argument("--graph", type=int, default=0, choices=(0, 1),
                    help="1: capture one stack step into a HIP graph and time its replays "
                         "(0: eager launches)")
    ap.add_argument("--streams", type=int, default=0, choices=(0, 1, 2),
                    help="2: each layer's backward-weight on a second stream, beside its "
                         "backward-data; 1: every pass on one stream; 0: time both after "
                         "the warm-up and keep the faster")
    ap.add_argument("--peaks", type=int, default=1, choices=(0, 1),
                    help="1: also measure the chip's reference points (fp32 matrix-core "
                         "loop, HBM copy, shader clock) and report them")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy 1 GiB device-to-device 3 times (HBM counter calibration)")
    return ap.parse_args()


def flops_of(L):
    if not hasattr(L, "K"):
        return 0.0  # pooling
    return 2.0 * L.N * L.K * L.P * L.Q * (L.C // L.group) * L.R * L.S


def bytes_of(L, p):
    """Compulsory HBM bytes of one pass (each tensor read or written once;
    pooling: x, y and the int32 mask forward, dy, mask and dx backward)."""
    if not hasattr(L, "K"):
        x, y = L.N * L.C * L.H * L.W, L.N * L.C * L.P * L.Q
        return 4.0 * (x + 2 * y)
    x = L.N * L.C * L.H * L.W
    y = L.N * L.K * L.P * L.Q
    w = L.K * (L.C // L.group) * L.R * L.S
    if p == "fwd":
        n = x + w + L.K + y
    elif p == "bwd_data":
        n = y + w + x
    else:
        n = x + y + w + L.K
    return 4.0 * n


class HipEvents:
    """Raw HIP events (for the library's timing hook)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                                 ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        e = ctypes.c_void_p()
        assert self.hip.hipEventCreate(ctypes.byref(e)) == 0
        return e

    def elapsed_ms(self, a, b):
        assert self.hip.hipEventSynchronize(b) == 0
        ms = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b) == 0
        return ms.value

    def destroy(self, e):
        self.hip.hipEventDestroy(e)


class LayerRun:
    """Device buffers and prepared library calls of one layer."""

    def __init__(self, cfg, li, L, stream, tune_reps=0):
        import numpy as np
        import torch
        import workloads
        import paper_1903_06934_amd as m

        self.L = L
        d = workloads.layer_inputs(cfg, li, L)
        dev = torch.device("cuda")
        t = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in d.items()}
        self.t = t
        self.y = torch.empty((L.N, L.K, L.P, L.Q), dtype=torch.float32, device=dev)
        self.dx = torch.empty((L.N, L.C, L.H, L.W), dtype=torch.float32, device=dev)
        self.dw = torch.empty_like(t["w"])
        self.db = torch.empty_like(t["b"])
        shape = L.shape
        self.ws = {}
        for pid in (0, 1, 2):
            n = m.workspace_size(pid, shape)
            self.ws[pid] = torch.empty(max(n, 256), dtype=torch.uint8, device=dev)
        if tune_reps > 0:
            self.tune(tune_reps)
        lib = m.lib()
        ws = lambda pid: (self.ws[pid].data_ptr(), self.ws[pid].numel())
        self.calls = {
            "fwd": (lib.conv_fwd, shape + (t["x"].data_ptr(), t["w"].data_ptr(),
                                           t["b"].data_ptr(), self.y.data_ptr()) + ws(0) + (stream,)),
            "bwd_data": (lib.conv_bwd_data, shape + (t["dy"].data_ptr(), t["w"].data_ptr(),
                                                     self.dx.data_ptr()) + ws(1) + (stream,)),
            "bwd_weight": (lib.conv_bwd_weight, shape + (t["x"].data_ptr(), t["dy"].data_ptr(),
                                                         self.dw.data_ptr(), self.db.data_ptr())
                           + ws(2) + (stream,)),
        }

    def tune(self, reps):
        """conv_tune every pass on this layer's tensors, with a workspace that
        fits every candidate; the library keeps the fastest plan per shape."""
        import torch
        import paper_1903_06934_amd as m
        shape, t = self.L.shape, self.t
        args = {0: (t["x"], t["w"], t["b"], self.y, None),
                1: (t["dy"], t["w"], None, self.dx, None),
                2: (t["x"], t["dy"], None, self.dw, self.db)}
        for pid in (0, 1, 2):
            n = m.plan_count(pid, shape)
            need = max(m.plan_workspace_size(pid, shape, i) for i in range(n))
            ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda")
            m.conv_tune(pid, shape, *args[pid], ws, reps=reps)
            self.ws[pid] = ws

    def plan(self, p):
        import paper_1903_06934_amd as m
        pid = PASSES.index(p)
        i = m.plan_get(pid, self.L.shape)
        return f"{i}: {m.plan_name(pid, self.L.shape, i)}"

    def run(self, p):
        fn, args = self.calls[p]
        st = fn(*args)
        if st != 0:
            import paper_1903_06934_amd as m
            raise m.MiconvError(st, f"{p} {self.L.name}")

    def bind_side(self, stream):
        """Also prepare the backward-weight call on a second stream (it has a
        workspace of its own, so it may run beside the other passes)."""
        fn, args = self.calls["bwd_weight"]
        self.side_calls = {"bwd_weight": (fn, args[:-1] + (stream,))}

    def run_side(self, p):
        fn, args = self.side_calls[p]
        st = fn(*args)
        if st != 0:
            import paper_1903_06934_amd as m
            raise m.MiconvError(st, f"{p} {self.L.name} (side stream)")


class PoolRun:
    """Device buffers and prepared library calls of one pooling layer; its
    passes are "fwd" and "bwd_data" (the input gradient)."""

    passes = ("fwd", "bwd_data")

    def __init__(self, cfg, li, L, stream):
        import numpy as np
        import torch
        import workloads
        import paper_1903_06934_amd as m

        self.L = L
        d = workloads.pool_inputs(cfg, li, L)
        dev = torch.device("cuda")
        self.x = torch.from_numpy(np.ascontiguousarray(d["x"])).to(dev)
        self.dy = torch.from_numpy(np.ascontiguousarray(d["dy"])).to(dev)
        self.y = torch.empty((L.N, L.C, L.P, L.Q), dtype=torch.float32, device=dev)
        self.mask = torch.empty((L.N, L.C, L.P, L.Q), dtype=torch.int32, device=dev)
        self.dx = torch.empty_like(self.x)
        lib = m.lib()
        mode = m.miconv.POOL_MODES[L.mode]
        geo = (mode,) + L.pshape
        self.calls = {
            "fwd": (lib.pool_fwd, geo + (self.x.data_ptr(), self.y.data_ptr(),
                                         self.mask.data_ptr(), stream)),
            "bwd_data": (lib.pool_bwd, geo + (self.dy.data_ptr(), self.mask.data_ptr(),
                                              self.dx.data_ptr(), stream)),
        }

    def plan(self, p):
        return f"{self.L.mode} pooling"

    def run(self, p):
        fn, args = self.calls[p]
        st = fn(*args)
        if st != 0:
            import paper_1903_06934_amd as m
            raise m.MiconvError(st, f"{p} {self.L.name}")


def stack_step(runs, side=None):
    """One training step's passes: forward over the layers, then backward in
    reverse.  With a side stream, each layer's backward-weight runs there,
    concurrently with its backward-data on the current stream: it starts once
    the layer's dy exists (after the forward half for the last layer, else
    after the backward-data of the layer above), and the step ends when both
    streams are done (the weight update of the next step needs every dw)."""
    import torch
    for r in runs:
        for _ in range(r.L.count):
            r.run("fwd")
    if side is None:
        for r in reversed(runs):
            for _ in range(r.L.count):
                if not isinstance(r, PoolRun):
                    r.run("bwd_weight")
                if not r.L.first:
                    r.run("bwd_data")
        return
    main = torch.cuda.current_stream()

    def handoff(src, dst):
        ev = torch.cuda.Event()
        ev.record(src)
        dst.wait_event(ev)

    handoff(main, side)
    for r in reversed(runs):
        for _ in range(r.L.count):
            if not isinstance(r, PoolRun):
                r.run_side("bwd_weight")
            if not r.L.first:
                r.run("bwd_data")
                handoff(main, side)
    handoff(side, main)


def time_call(fn, reps, flush_buf=None):
    """Median and min device ms of fn() over reps, torch events on the
    current stream (the stream the library launches on)."""
    import torch
    ts = []
    for _ in range(reps):
        if flush_buf is not None:
            flush_buf.add_(1.0)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        ts.append(a.elapsed_time(b))
    return statistics.median(ts), min(ts)


def kernel_time(run, p, reps, hev):
    """Average device ms of the pass's GEMM kernel(s) alone, from the
    library's timing hook (events recorded around the GEMM launches)."""
    import torch
    import paper_1903_06934_amd as m
    lib = m.lib()
    a, b = hev.create(), hev.create()
    ts = []
    try:
        assert lib.conv_set_timing_events(a, b) == 0
        for _ in range(reps):
            run.run(p)
            ts.append(hev.elapsed_ms(a, b))
    finally:
        lib.conv_set_timing_events(None, None)
        torch.cuda.synchronize()
        hev.destroy(a)
        hev.destroy(b)
    return sum(ts) / len(ts)


TRAFFIC_DIR = os.path.join(ROOT, "profiles")
KERNEL_SOURCE = os.path.join(ROOT, "paper_1903_06934_amd", "csrc", "conv_kernels.hip")


def measured_traffic(cfg, layer, p, plan):
    """HBM bytes per launch of the (cfg, layer, pass) GEMM from a committed
    rocprofv3 counter summary (profiles/traffic_*.txt), if one exists for
    exactly this workload and plan and the kernel source has not changed
    since."""
    import glob
    import hashlib
    sha = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    for f in sorted(glob.glob(os.path.join(TRAFFIC_DIR, "traffic_*.txt"))):
        kv = {}
        for line in open(f):
            if ":" in line and not line.startswith(("#", " ")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
        if (kv.get("workload") == f"{cfg}:{layer}:{p}" and kv.get("kernel_source_sha256") == sha
                and kv.get("plan") == plan and "traffic_bytes_per_launch" in kv):
            return float(kv["traffic_bytes_per_launch"])
    return None


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, layers, target_s):
    """The oracle (fp64 loop nests, all host threads) on a batch slice of
    the same stack: images/s on the host, and GFLOP/s per layer and pass."""
    import oracle
    import workloads
    o = oracle.default()

    def run_stack(n):
        secs, per = 0.0, []
        for li, L in enumerate(layers):
            Ls = L.with_batch(n)
            d = workloads.layer_inputs(cfg, li, Ls)
            calls = [("fwd", lambda: o.conv_fwd(Ls.shape, d["x"], d["w"], d["b"])),
                     ("bwd_weight", lambda: o.conv_bwd_weight(Ls.shape, d["x"], d["dy"]))]
            if not L.first:
                calls.append(("bwd_data", lambda: o.conv_bwd_data(Ls.shape, d["dy"], d["w"])))
            for p, fn in calls:
                t0 = time.perf_counter()
                fn()
                dt = time.perf_counter() - t0
                secs += dt * L.count
                per.append({"layer": L.name, "pass": p,
                            "gflops": round(flops_of(Ls) / dt / 1e9, 3)})
        return secs, per

    # Calibrate on one image, then size the sample to the target time.
    t1, per = run_stack(1)
    n = max(1, min(layers[0].N, int(target_s / max(t1, 1e-6))))
    secs = t1
    if n > 1:
        secs, per = run_stack(n)
    return {"value": n / secs, "unit": "img/s", "cores": o.num_threads(), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"the same stack at batch {n} of {layers[0].N}, every layer and pass "
                      f"(fp64 direct loop nests; input generation not timed), {secs:.1f} s; "
                      "img/s is exact for the full batch since every pass is linear in it",
            "per_layer_gflops": per}


def measured_peaks():
    """The chip's reference points next to the datasheet peaks: a
    register-only fp32 matrix-core loop at 1, 2 and 4 waves per SIMD (with
    the shader clock it ran at), and a 1 GiB device copy."""
    import torch
    from paper_1903_06934_amd import peaks
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    mfma = {}
    for wps in (1, 2, 4):
        tf, ghz = peaks.mfma_f32(wps, cus)
        mfma[f"{wps}_waves_per_simd"] = {"tflops": round(tf, 1), "shader_ghz": round(ghz, 3)}
    gbs, ok = peaks.copy_gbs()
    if not ok:
        raise RuntimeError("peak_copy produced a wrong copy")
    return {"compute_units": cus,
            "mfma_f32_16x16x4_loop": mfma,
            "hbm_copy_gbs": round(gbs, 1),
            "note": "register-only v_mfma_f32_16x16x4f32 loop with 8 independent chains per "
                    "wave; copy of 1 GiB by a float4 kernel, read + write bytes over time"}


def bench_config(cfg, args, with_cpu):
    import contextlib
    import torch
    # A graph is captured on a side stream (the legacy stream cannot
    # capture), so then every launch of the run goes there.
    side = torch.cuda.Stream() if args.graph else None
    with torch.cuda.stream(side) if side is not None else contextlib.nullcontext():
        return _bench_config(cfg, args, with_cpu)


def _bench_config(cfg, args, with_cpu):
    import torch
    import workloads

    name, layers = workloads.config(cfg)
    stream = torch.cuda.current_stream().cuda_stream
    runs = [PoolRun(cfg, li, L, stream) if isinstance(L, workloads.PoolLayer)
            else LayerRun(cfg, li, L, stream, args.tune) for li, L in enumerate(layers)]
    side_stream = torch.cuda.Stream() if args.streams != 1 else None
    if side_stream is not None:
        for r in runs:
            if isinstance(r, LayerRun):
                r.bind_side(side_stream.cuda_stream)
    torch.cuda.synchronize()
    N = layers[0].N

    def timed_steps(side, k):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(k):
            stack_step(runs, side)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / k

    side = side_stream if args.streams == 2 else None
    for _ in range(args.warmup):
        stack_step(runs, side)
    torch.cuda.synchronize()
    schedule_ms = None
    if args.streams == 0:
        # Time both schedules (alternating, best of two rounds) and keep the
        # faster for the timed region.
        k = max(3, min(10, args.steps // 2))
        one, two = [], []
        for _ in range(2):
            one.append(timed_steps(None, k))
            two.append(timed_steps(side_stream, k))
        schedule_ms = {"one_stream": round(min(one), 4), "two_streams": round(min(two), 4)}
        side = side_stream if min(two) < min(one) else None
    step = lambda: stack_step(runs, side)  # noqa: E731
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=torch.cuda.current_stream()):
            stack_step(runs, side)
        graph.replay()
        torch.cuda.synchronize()
        step = graph.replay
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    step_ms = e0.elapsed_time(e1) / args.steps

    flush = torch.empty(128 << 20, dtype=torch.float32, device="cuda")
    ridge = PEAK_TFLOPS * 1e12 / (PEAK_GBS * 1e9)
    per = []
    tot = {p: [0.0, 0.0] for p in PASSES}
    for r in runs:
        L = r.L
        for p in getattr(r, "passes", PASSES):
            med, mn = time_call(lambda: r.run(p), args.reps)
            F = flops_of(L)
            B = bytes_of(L, p)
            t_roof = max(F / (PEAK_TFLOPS * 1e12), B / (PEAK_GBS * 1e9)) * 1e3
            in_stack = not (p == "bwd_data" and L.first)
            row = {"layer": L.name, "pass": p, "count": L.count, "in_stack": in_stack,
                   "cache": "warm", "ms": round(med, 4), "ms_min": round(mn, 4),
                   "tflops": round(F / med / 1e9, 2), "gbs": round(B / med / 1e6, 1),
                   "roof_frac": round(t_roof / med, 3), "plan": r.plan(p)}
            if args.flush or F < 2 * ridge * B:
                # Memory-bound or near the ridge: also from cold caches.
                cmed, _ = time_call(lambda: r.run(p), args.reps, flush)
                row.update({"ms_cold": round(cmed, 4), "gbs_cold": round(B / cmed / 1e6, 1),
                            "roof_frac_cold": round(t_roof / cmed, 3)})
            per.append(row)
            if in_stack and F > 0:
                tot[p][0] += F * L.count
                tot[p][1] += med * L.count
    del flush

    # Dominant kernel: the GEMM of the (layer, pass) with the largest share
    # of the step.
    dom = max((x for x in per if x["in_stack"] and x["tflops"] > 0),
              key=lambda x: x["ms"] * x["count"])
    hev = HipEvents()
    drun = next(r for r in runs if r.L.name == dom["layer"])
    k_ms = kernel_time(drun, dom["pass"], args.reps, hev)
    F = flops_of(drun.L)
    ai = F / bytes_of(drun.L, dom["pass"])
    if ai >= ridge:
        ach = F / k_ms / 1e9
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_TFLOPS, 4), "traffic": None}
    else:
        ach = bytes_of(drun.L, dom["pass"]) / k_ms / 1e6
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_GBS,
                "unit": "GB/s", "frac": round(ach / PEAK_GBS, 4), "traffic": None}
    roof["traffic"] = measured_traffic(cfg, dom["layer"], dom["pass"], dom["plan"])
    roof.update({"kernel": f"{dom['pass']} GEMM of {dom['layer']} ({dom['plan']})",
                 "kernel_ms": round(k_ms, 4), "flops_per_launch": F,
                 "bytes_per_launch": bytes_of(drun.L, dom["pass"])})

    line = {
        "metric": METRIC,
        "value": round(N * args.steps / (step_ms * args.steps / 1e3), 2),
        "unit": "img/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": WORKLOAD_NAMES[cfg], "name": name, "global_batch": N,
                   "layers": len(layers), "parallelism": "single GPU",
                   "launch": ("hip graph" if args.graph else "eager") +
                   (", backward-weight on a second stream" if side is not None
                    else ", one stream")},
        "tflops_per_pass": {p: round(tot[p][0] / tot[p][1] / 1e9, 2) if tot[p][1] else None
                            for p in PASSES},
        "stack_tflops": round(sum(v[0] for v in tot.values()) / (step_ms * 1e9), 2),
        "roofline": roof,
        "per_layer": per,
    }
    if schedule_ms is not None:
        line["schedule_ms_per_step"] = schedule_ms
    if args.peaks:
        line["measured_peaks"] = measured_peaks()
    if with_cpu:
        line["cpu_baseline"] = cpu_baseline(cfg, layers, args.cpu_seconds)
    del runs
    torch.cuda.empty_cache()
    return line


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU "
              "data-parallel path is a design, not part of this build.", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    import paper_1903_06934_amd as m
    m.lib()
    if args.copy_calibration:
        x = torch.ones(1 << 28, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print("copied 1 GiB device-to-device 3 times", flush=True)
        return
    if args.profile_pass:
        import workloads
        cfg, lname, p = args.profile_pass.split(":")
        cfg = int(cfg)
        layers = workloads.config(cfg)[1]
        li = [L.name for L in layers].index(lname)
        if args.plan is not None:
            m.plan_set(PASSES.index(p), layers[li].shape, args.plan)
        run = LayerRun(cfg, li, layers[li], torch.cuda.current_stream().cuda_stream,
                       0 if args.plan is not None else args.tune)
        for _ in range(args.reps):
            run.run(p)
        torch.cuda.synchronize()
        print(f"ran {args.profile_pass} x{args.reps} with plan: {run.plan(p)}", flush=True)
        return
    cfgs = [0, 1, 2, 3, 4, 5] if args.config == "all" else [int(args.config)]
    for cfg in cfgs:
        line = bench_config(cfg, args, with_cpu=args.cpu_seconds > 0 and cfg == cfgs[0])
        print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
