#!/usr/bin/env python3
"""Benchmark of the SS2D selective-scan path on one MI355X.

Workload: VMamba-T stage 1, batch 1, 56x56 feature map (L = 3136), K = 4
directions, 192 channels, N = 16 states, fp32, seeded synthetic inputs
(workloads.STAGE1).

A step is one SS2D forward of the whole path, x [1, 192, 56, 56] -> y of the
same shape: cross-scan fused into the scan's loads, the scan, and the
cross-merge, via one vmb_selective_scan_fwd call in the 2-D layout (full
variant). The same step with vmb_mean_scan_fwd (VMeanba) is timed next to it.
Inputs are resident in HBM before timing starts; each step reads a different
copy of the inputs (rotation over enough copies to exceed the 256 MB Infinity
Cache), so every step streams from HBM.

Prints one JSON line (rank 0). The `roofline` object covers the dominant
kernel, the full scan, timed alone on the sequence layout with HIP events on
its stream, against the published MI355X peaks: HBM 8 TB/s (algorithmic bytes:
u, delta, B, C read once, y written once) and fp32 vector 157.3 TFLOP/s (7 FLOP
per (channel, state, position): Delta*A, exp, Delta*u*B, state FMA, output
FMA). `bound` names the roof the kernel comes closer to; the other one is
reported next to it. `traffic` is the HBM bytes per launch measured with
rocprofv3 counters (profiles/), reported only while the kernel sources still
match the ones profiled. `roofline.step` does the same for the whole timed
step (2-D layout: the scan and the merge). `cpu_baseline` times the fp64
oracle on the host (full and mean SS2D forwards, one-thread times, a sampled
batched workload) and `accuracy` compares the GPU outputs of the timed step
with it.

--calibrate runs a plain 256 MiB device copy first, the reference dispatch the
counter runs scale FETCH_SIZE / WRITE_SIZE by.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402

HBM_PEAK_GBPS = 8000.0
FP32_VECTOR_PEAK_TFLOPS = 157.3  # MI355X published fp32 vector peak (packed FMA)
# per (channel, state, position): Delta*A, exp, Delta*u*B, state FMA, output FMA
FLOP_PER_ELEM = 7
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "full_scan_seq_56x56_c192_n16_traffic.txt")
STEP_FILE = os.path.join(ROOT, "profiles", "ss2d_step_56x56_c192_n16_traffic.txt")
# the sources the profiled kernels are compiled from
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2412_16602_amd", "csrc", f)
                  for f in ("scan_chunked.hip", "vmb_device.h")]
STEP_SOURCES = [os.path.join(ROOT, "paper_2412_16602_amd", "csrc", f)
                for f in ("scan_chunked.hip", "vmb_device.h", "cross.hip", "scan_full.hip")]
METRIC = ("SS2D selective-scan µs/call + HBM GB/s (% peak), full vs mean, "
          "VMamba-T 56×56")
ROTATE_BYTES = 768 << 20  # > 2x the 256 MB MALL
MFMA_F32_PEAK_TFLOPS = 157.3  # dense fp32 matrix-core peak


def seq_bytes(s: workloads.Shape, batch: int, esz_in=4, esz_out=4) -> int:
    """Algorithmic bytes of one scan call, sequence layout: u, delta, B, C read
    once, y written once (A, D, dt_bias included)."""
    K, Dc, L, N = 4, s.channels, s.L, s.N
    return (2 * batch * K * Dc * L + 2 * batch * K * N * L) * esz_in + batch * K * Dc * L * esz_out \
        + (K * Dc * N + 2 * K * Dc) * 4


def ss2d_bytes(s: workloads.Shape, batch: int, esz_in=4, esz_out=4) -> int:
    """Algorithmic bytes of one SS2D forward, 2-D layout: x read once, delta,
    B, C read once, merged y written once."""
    K, Dc, L, N = 4, s.channels, s.L, s.N
    return (batch * Dc * L + batch * K * Dc * L + 2 * batch * K * N * L) * esz_in \
        + batch * Dc * L * esz_out + (K * Dc * N + 2 * K * Dc) * 4


def gpu_bench(args):
    import torch

    from paper_2412_16602_amd import vmb

    dev = torch.device("cuda:0")
    shape = workloads.STAGE1
    stream = torch.cuda.current_stream()

    def upload(inp, layout):
        g = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        u = g(inp.x if layout == "2d" else inp.u)
        return dict(u=u, delta=g(inp.delta), A=g(inp.A), B=g(inp.B), C=g(inp.C), D=g(inp.D),
                    dt_bias=g(inp.dt_bias))

    inp2d = workloads.make_inputs(shape, "2d")
    inpseq = workloads.make_inputs(shape, "seq")
    step_bytes = ss2d_bytes(shape, shape.batch)
    scan_bytes = seq_bytes(shape, shape.batch)
    n_rot = max(2, -(-ROTATE_BYTES // step_bytes))

    def make_sets(inp, layout, variant, n):
        base = upload(inp, layout)
        out_shape = tuple(inp.x.shape) if layout == "2d" else tuple(inp.delta.shape)
        lay = vmb.VMB_LAYOUT_2D if layout == "2d" else vmb.VMB_LAYOUT_SEQ
        need = vmb.vmb_scan_workspace_bytes(variant == "mean", shape.batch, 4, shape.channels,
                                            shape.L, shape.N, lay)
        sets = []
        for i in range(n):
            d = {k: (v.clone() if i else v) for k, v in base.items()}
            d["y"] = torch.empty(out_shape, dtype=torch.float32, device=dev)
            d["ws"] = torch.empty(max(need, 1), dtype=torch.uint8, device=dev) if need else None
            sets.append(d)
        return sets, lay

    def runner(variant, sets, lay):
        fn = vmb.vmb_selective_scan_fwd if variant == "full" else vmb.vmb_mean_scan_fwd

        def call(i):
            d = sets[i % len(sets)]
            fn(d["u"], d["delta"], d["A"], d["B"], d["C"], d["D"], d["dt_bias"], True, d["y"],
               layout=lay, workspace=d["ws"], stream=stream)
        return call

    # The stream is idle after the synchronize that ends the warmup. With
    # nothing queued ahead of the start event, the host-side marshalling and
    # launch of the first timed call (about 15 us on the GPU host, against
    # about 25 us of device time per call) would be timed as device idle: a
    # 20-step run read 27.1 us per call where 200 steps read 25.9. A device
    # sleep of about 60 us is queued before the start event, so the timed
    # region starts with the first calls already queued; the later calls are
    # still enqueued at the host's own rate, so a host slower than the device
    # would still show in the result.
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    probe = 1 << 20
    torch.cuda._sleep(probe)  # first use (module load) outside the measurement
    torch.cuda.synchronize()
    e0.record(stream)
    torch.cuda._sleep(probe)
    e1.record(stream)
    torch.cuda.synchronize()
    lead_cycles = max(1, int(probe * 60.0 / (e0.elapsed_time(e1) * 1e3)))

    def timed(call, steps, warmup):
        for i in range(warmup):
            call(i)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(lead_cycles)
        e0.record(stream)
        for i in range(steps):
            call(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / steps  # us per call

    def per_call(call, n):
        """Each call bracketed by its own events: p10 / median / p90 in us."""
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(n)]
        for i, (a, b) in enumerate(ev):
            a.record(stream)
            call(i)
            b.record(stream)
        torch.cuda.synchronize()
        t = np.array([a.elapsed_time(b) * 1e3 for a, b in ev])
        return {"p10": round(float(np.percentile(t, 10)), 3),
                "p50": round(float(np.percentile(t, 50)), 3),
                "p90": round(float(np.percentile(t, 90)), 3)}

    res = {}
    outputs = {}
    # --- the step: SS2D forward, 2-D layout, full and mean
    for variant in ("full", "mean"):
        sets, lay = make_sets(inp2d, "2d", variant, n_rot)
        call = runner(variant, sets, lay)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        us = timed(call, args.steps, args.warmup)
        wall = time.perf_counter() - t0
        warm = timed(runner(variant, sets[:1], lay), args.steps, 2)
        dist = per_call(call, min(args.steps, 100))
        res[f"ss2d_{variant}"] = dict(us=us, warm_us=warm, wall_s=wall, dist=dist)
        torch.cuda.synchronize()
        outputs[variant] = sets[0]["y"].cpu().numpy()  # set 0: the workload's own inputs
        del sets
    # --- dominant kernel alone: the scan, sequence layout (one kernel per call for full)
    for variant in ("full", "mean"):
        n = max(2, -(-ROTATE_BYTES // scan_bytes))
        sets, lay = make_sets(inpseq, "seq", variant, n)
        us = timed(runner(variant, sets, lay), args.steps, args.warmup)
        res[f"seq_{variant}"] = dict(us=us)
        del sets
    torch.cuda.synchronize()
    return res, step_bytes, scan_bytes, n_rot, outputs


def source_hash(paths=None) -> str:
    import hashlib
    h = hashlib.sha256()
    for path in (KERNEL_SOURCES if paths is None else paths):
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def profile_values(path, sources):
    """The machine-read lines ("key: value") of a committed counter summary,
    or None if absent or taken on other kernel sources."""
    try:
        with open(path) as f:
            kv = dict(line.split(":", 1) for line in f if ":" in line)
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("kernel_sources_sha256_16") != source_hash(sources):
        return None
    return kv


def measured_traffic():
    """HBM bytes per launch of the full scan from the committed counter
    summary, or None."""
    kv = profile_values(TRAFFIC_FILE, KERNEL_SOURCES)
    try:
        return int(kv["traffic_bytes_per_launch"]) if kv else None
    except (KeyError, ValueError):
        return None


def measured_step():
    """Kernel-trace time and counter bytes of the whole 2-D step (all its
    kernels) from the committed summary, or None."""
    kv = profile_values(STEP_FILE, STEP_SOURCES)
    if not kv:
        return None
    try:
        return {"kernels_us": float(kv["step_kernels_us"]),
                "counter_bytes": int(kv["step_traffic_bytes"]),
                "kernels": kv.get("step_kernels", "")}
    except (KeyError, ValueError):
        return None


def calibrate_copy():
    """A plain streaming kernel of known size: 256 MiB read, 256 MiB written
    (an elementwise negation, so it shows up as its own kernel)."""
    import torch
    src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst


def _timed_reps(fn, budget_s: float, max_reps: int = 1000):
    """Run fn() until about budget_s seconds have passed; mean seconds per call."""
    reps, total = 0, 0.0
    while True:
        t0 = time.perf_counter()
        fn()
        total += time.perf_counter() - t0
        reps += 1
        if total >= budget_s or reps >= max_reps:
            return total / reps, reps


def cpu_baseline(budget_s: float, gpu_out=None):
    """The fp64 oracle on the host, in bounded samples (about budget_s seconds
    each for the two main lines, less for the others):
      - one SS2D forward (cross-scan, full scan, merge) at the bench workload,
        every available core; this is `value`;
      - the same forward with the mean (VMeanba) scan;
      - one-thread full forwards of the tiny 7x7 workload and the stage-1 one;
      - a sampled batched workload: one batch item of the batch-128 bf16
        stage-1 workload (items are independent), scaled to the batch.
    With gpu_out (the GPU outputs of the timed step on its first input set),
    also the elementwise error of those outputs against the oracle."""
    import oracle

    threads = len(os.sched_getaffinity(0))
    threads = min(threads, int(os.environ.get("OMP_NUM_THREADS", threads)))
    inp = workloads.make_inputs(workloads.STAGE1, "2d")
    H, W = inp.shape.H, inp.shape.W

    def forward(variant, x_inp, nthreads):
        xs = oracle.cross_scan(x_inp.x)
        fn = oracle.full_scan if variant == "full" else oracle.mean_scan
        ys = fn(xs, x_inp.delta, x_inp.A, x_inp.B, x_inp.C, x_inp.D, x_inp.dt_bias, True,
                nthreads=nthreads)
        return oracle.cross_merge(np.ascontiguousarray(ys), x_inp.shape.H, x_inp.shape.W, "f64")

    full_s, full_n = _timed_reps(lambda: forward("full", inp, threads), budget_s)
    mean_s, mean_n = _timed_reps(lambda: forward("mean", inp, threads), budget_s / 2)
    tiny = workloads.make_inputs(workloads.TINY, "2d")
    tiny_s, tiny_n = _timed_reps(lambda: forward("full", tiny, 1), 1.0)
    one_s, one_n = _timed_reps(lambda: forward("full", inp, 1), budget_s / 2, max_reps=3)
    # one batch item of the batch-128 bf16 workload, drawn with its own recipe
    big = workloads.make_inputs(workloads.BATCHED_BF16, "2d", batch=1)
    big_s, big_n = _timed_reps(lambda: forward("full", big, threads), budget_s / 4, max_reps=20)
    res = dict(value=full_s * 1e6, unit="us/call", cores=threads, kind="oracle",
               sample=f"{full_n} x one SS2D forward (cross-scan, full scan, merge) at 1x56x56, "
                      f"192 channels, N=16, fp64, {threads} threads",
               cpu_model=cpu_model(),
               mean_us=round(mean_s * 1e6, 1),
               mean_sample=f"{mean_n} x the same forward with the VMeanba mean scan",
               single_thread_us={"tiny_7x7_c32_n4_full": round(tiny_s * 1e6, 1),
                                 "stage1_56x56_c192_n16_full": round(one_s * 1e6, 1)},
               batched_sample={"workload": workloads.BATCHED_BF16.name,
                               "sample": f"{big_n} x one of 128 batch items (independent), "
                                         f"{threads} threads",
                               "us_per_item": round(big_s * 1e6, 1),
                               "us_whole_batch_scaled": round(big_s * 1e6 * 128, 1)})
    acc = None
    if gpu_out is not None:
        acc = {}
        for variant in ("full", "mean"):
            if variant not in gpu_out:
                continue
            ref = forward(variant, inp, threads)
            got = np.asarray(gpu_out[variant], dtype=np.float64)
            err = np.abs(got - ref)
            acc[variant] = {"max_abs_err": float(err.max()),
                            "max_rel_err": float((err / np.maximum(np.abs(ref), 1e-30)).max()),
                            "worst_vs_fp32_tol": float((err / (1e-5 + 1e-4 * np.abs(ref))).max())}
    return res, acc


# The paper's Table 1 times of the original (all-channel) kernel on its own
# GPU (an NVIDIA RTX A6000), in ms, for context only.
PAPER_TABLE1_MS = {("tiny_small", 384, 3136): 5.46, ("tiny_small", 768, 784): 2.23,
                   ("tiny_small", 1536, 196): 1.10, ("tiny_small", 3072, 49): 0.71,
                   ("base", 512, 3136): 5.86, ("base", 1024, 784): 2.94,
                   ("base", 2048, 196): 1.47, ("base", 4096, 49): 0.93}


def table1_bench(steps: int, warmup: int):
    """The decomposition of the paper's kernel experiments (Table 1 shapes,
    batch 128, one state): the scan on materialised inputs over all channels,
    and the VMeanba path (T on both inputs, then the scan at one channel).
    Inputs are drawn on the GPU with the distributions of
    workloads.make_discrete_inputs (uniform decays, low cross-channel
    variance bu, normal C); the one-channel scan reads the reduced inputs
    the reduce has just written, as it would in use."""
    import torch

    from paper_2412_16602_amd import vmb

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    g = torch.Generator(device=dev)
    g.manual_seed(1)
    B = workloads.TABLE1_BATCH

    def timed(fn):
        """us per call: `steps` calls captured in one HIP graph and replayed,
        so the host's per-call launch cost (larger than the one-channel
        kernel itself) stays out of the kernel time."""
        for _ in range(warmup):
            fn(stream)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cap = torch.cuda.current_stream()
            for _ in range(steps):
                fn(cap)
        graph.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        del graph
        return e0.elapsed_time(e1) * 1e3 / steps

    rows = []
    for backbone, D, L in workloads.TABLE1_SHAPES:
        # enough input sets, used in turn, that each call reads from HBM
        # rather than the 256 MB MALL
        set_bytes = B * D * L * 12
        n_sets = max(2, -(-ROTATE_BYTES // set_bytes))
        sets = []
        lo, hi = math.exp(-0.1), math.exp(-0.001)
        for _ in range(n_sets):
            # the distributions of workloads.make_discrete_inputs
            abar = lo + (hi - lo) * torch.rand(B, D, L, device=dev, generator=g)
            base = torch.randn(B, 1, L, device=dev, generator=g)
            bu = 0.05 * (base + 0.1 * torch.randn(B, D, L, device=dev, generator=g))
            sets.append((abar, bu, torch.empty_like(abar)))
        C = torch.randn(B, L, device=dev, generator=g)
        am = torch.empty(B, 1, L, device=dev)
        bm = torch.empty(B, 1, L, device=dev)
        y1 = torch.empty(B, 1, L, device=dev)
        turn = [0]

        def nxt():
            turn[0] = (turn[0] + 1) % n_sets
            return sets[turn[0]]

        def full(st):
            abar, bu, y = nxt()
            vmb.vmb_discrete_scan(abar, bu, C, None, y, stream=st)

        def reduce(st):
            abar, bu, _ = nxt()
            vmb.vmb_channel_mean(abar, am.view(B, L), stream=st)
            vmb.vmb_channel_mean(bu, bm.view(B, L), stream=st)

        full_us = timed(full)
        red_us = timed(reduce)
        d1_us = timed(lambda st: vmb.vmb_discrete_scan(am, bm, C, None, y1, stream=st))
        full_bytes = B * D * L * 12 + B * L * 4
        red_bytes = 2 * (B * D * L * 4 + B * L * 4)
        rows.append({
            "backbone": backbone, "channels": D, "L": L, "batch": B,
            "full_us": round(full_us, 2),
            "full_gbps": round(full_bytes / (full_us * 1e-6) / 1e9, 1),
            "full_hbm_frac": round(full_bytes / (full_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            "mean_scan_d1_us": round(d1_us, 2),
            "speedup_scan": round(full_us / d1_us, 1),
            "mean_reduce_us": round(red_us, 2),
            "reduce_gbps": round(red_bytes / (red_us * 1e-6) / 1e9, 1),
            "paper_original_ms_a6000": PAPER_TABLE1_MS[(backbone, D, L)],
        })
        del sets, C, am, bm, y1
        torch.cuda.empty_cache()
    return {"metric": "one-state scan on materialised inputs, Table 1 shapes (us/call)",
            "unit": "us/call", "dtype": "f32", "data": "synthetic",
            "timing": f"HIP graph of {steps} calls replayed, events on the replay stream",
            "rows": rows}


def variants_bench(steps: int, warmup: int):
    """The mean scan's reading variants (vmb_mean_scan_fwd_ex options) and the
    zero-order-hold B of both scans at the stage-1 workload, next to the main
    reading: µs per call, inputs rotated past the MALL, events on the launch
    stream."""
    import torch

    from paper_2412_16602_amd import vmb

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    shape = workloads.STAGE1
    opts = {"main": 0, "skip_per_channel": vmb.VMB_MEAN_SKIP_PER_CHANNEL, "raw": vmb.VMB_MEAN_RAW,
            "no_broadcast": vmb.VMB_MEAN_NO_BROADCAST,
            "raw_no_broadcast": vmb.VMB_MEAN_RAW | vmb.VMB_MEAN_NO_BROADCAST,
            "pooled": vmb.VMB_MEAN_POOLED,
            "zoh": vmb.VMB_SCAN_ZOH,
            # the full scan, first-order and zero-order-hold B (no T)
            "full_first_order": ("full", 0), "full_zoh": ("full", vmb.VMB_SCAN_ZOH)}
    rows = []
    for layout in ("seq", "2d"):
        inp = workloads.make_inputs(shape, layout)
        g = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        lay = vmb.VMB_LAYOUT_2D if layout == "2d" else vmb.VMB_LAYOUT_SEQ
        base = dict(u=g(inp.x if layout == "2d" else inp.u), delta=g(inp.delta), A=g(inp.A),
                    B=g(inp.B), C=g(inp.C), D=g(inp.D), dt_bias=g(inp.dt_bias))
        nbytes = ss2d_bytes(shape, shape.batch) if layout == "2d" else seq_bytes(shape, shape.batch)
        n = max(2, -(-ROTATE_BYTES // nbytes))
        need = max(vmb.vmb_scan_workspace_bytes(v, shape.batch, 4, shape.channels, shape.L,
                                                shape.N, lay) for v in (0, 1))
        sets = [{k: (v.clone() if i else v) for k, v in base.items()} for i in range(n)]
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
        for name, opt in opts.items():
            full = isinstance(opt, tuple)
            if full:
                opt = opt[1]
            if layout == "2d" and not full and opt & vmb.VMB_MEAN_NO_BROADCAST:
                continue
            if layout == "2d":
                yshape = tuple(inp.x.shape)
            else:
                yshape = tuple(inp.delta.shape)
                if not full and opt & vmb.VMB_MEAN_NO_BROADCAST:
                    yshape = yshape[:2] + (1,) + yshape[3:]
            ys = [torch.empty(yshape, device=dev) for _ in range(n)]

            fn = vmb.vmb_selective_scan_fwd_ex if full else vmb.vmb_mean_scan_fwd_ex

            def call(i):
                d = sets[i % n]
                fn(d["u"], d["delta"], d["A"], d["B"], d["C"], d["D"], d["dt_bias"], True,
                   ys[i % n], opt, layout=lay, workspace=ws, stream=stream)
            for i in range(warmup):
                call(i)
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for i in range(steps):
                call(i)
            e1.record(stream)
            torch.cuda.synchronize()
            rows.append({"layout": layout, "reading": name, "options": opt,
                         "us": round(e0.elapsed_time(e1) * 1e3 / steps, 3)})
            del ys
        del sets, ws
        torch.cuda.empty_cache()
    return {"metric": "VMeanba reading variants and zero-order-hold B, stage-1 56x56 c192 N16 fp32 "
                      "(us/call)",
            "unit": "us/call", "dtype": "f32", "data": "synthetic", "rows": rows}


def workloads_bench(steps: int, warmup: int):
    """Full and mean scans at every N = 16 workload (the stage-1 map, the
    batch-32 later stages, batch-128 bf16, the high-resolution map), both
    layouts: us per call with HIP events on the launch stream. Inputs are
    drawn on the GPU with the distributions of workloads.make_inputs
    (channel-shared base plus 0.05 noise, delta ~ N(0, 0.5), softplus(dt_bias)
    log-uniform on [1e-3, 1e-1], B, C ~ N(0, 1), A = -(n + 1), D = 1; bf16
    workloads round the streamed tensors), because the host generator takes
    minutes at the batch-128 size; enough input sets are used in turn that
    every call reads from HBM rather than the 256 MB MALL."""
    import torch

    from paper_2412_16602_amd import vmb

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    g = torch.Generator(device=dev)
    g.manual_seed(2)
    rows = []
    for shp in (workloads.STAGE1, workloads.STAGE2, workloads.STAGE3, workloads.STAGE4,
                workloads.BATCHED_BF16, workloads.HIRES):
        b, K, Dc, L, N, H, W = shp.batch, 4, shp.channels, shp.L, shp.N, shp.H, shp.W
        bf16 = shp.dtype == "bf16"
        dt = torch.bfloat16 if bf16 else torch.float32
        esz = 2 if bf16 else 4
        A = -torch.arange(1, N + 1, device=dev, dtype=torch.float32).repeat(K * Dc, 1)
        D = torch.ones(K * Dc, device=dev)
        lo, hi = math.log(1e-3), math.log(1e-1)
        dtv = torch.exp(torch.empty(K * Dc, device=dev).uniform_(lo, hi, generator=g))
        dt_bias = torch.log(torch.expm1(dtv))
        for layout in ("seq", "2d"):
            lay = vmb.VMB_LAYOUT_2D if layout == "2d" else vmb.VMB_LAYOUT_SEQ
            nbytes = ss2d_bytes(shp, b, esz, esz) if layout == "2d" else seq_bytes(shp, b, esz, esz)
            n_sets = max(1, min(8, -(-ROTATE_BYTES // nbytes)))

            def draw():
                if layout == "2d":
                    u = torch.randn(b, 1, H, W, device=dev, generator=g) + \
                        0.05 * torch.randn(b, Dc, H, W, device=dev, generator=g)
                else:
                    u = torch.randn(b, K, 1, L, device=dev, generator=g) + \
                        0.05 * torch.randn(b, K, Dc, L, device=dev, generator=g)
                delta = math.sqrt(0.5) * torch.randn(b, K, Dc, L, device=dev, generator=g)
                Bm = torch.randn(b, K, N, L, device=dev, generator=g)
                Cm = torch.randn(b, K, N, L, device=dev, generator=g)
                return [t.to(dt).contiguous() for t in (u, delta, Bm, Cm)]

            sets = [draw() for _ in range(n_sets)]
            yshape = (b, Dc, H, W) if layout == "2d" else (b, K, Dc, L)
            y = torch.empty(yshape, device=dev, dtype=dt)
            for variant in ("full", "mean"):
                fn = vmb.vmb_selective_scan_fwd if variant == "full" else vmb.vmb_mean_scan_fwd
                need = vmb.vmb_scan_workspace_bytes(variant == "mean", b, K, Dc, L, N, lay)
                ws = torch.empty(need, dtype=torch.uint8, device=dev) if need else None

                def call(i):
                    u, delta, Bm, Cm = sets[i % n_sets]
                    fn(u, delta, A, Bm, Cm, D, dt_bias, True, y, layout=lay, workspace=ws,
                       stream=stream)
                # about 0.2 s of calls per measurement
                for i in range(warmup):
                    call(i)
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                call(0)
                e1.record(stream)
                torch.cuda.synchronize()
                n = max(3, min(steps, int(0.2e6 / max(1.0, e0.elapsed_time(e1) * 1e3))))
                e0.record(stream)
                for i in range(n):
                    call(i)
                e1.record(stream)
                torch.cuda.synchronize()
                us = e0.elapsed_time(e1) * 1e3 / n
                elems = b * K * Dc * N * L
                rows.append({"workload": shp.name, "layout": layout, "variant": variant,
                             "dtype": shp.dtype, "us": round(us, 2), "calls": n,
                             "gbps": round(nbytes / (us * 1e-6) / 1e9, 1),
                             "hbm_frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                             "alu_frac": round(elems * FLOP_PER_ELEM / (us * 1e-6) / 1e12
                                               / FP32_VECTOR_PEAK_TFLOPS, 4)
                             if variant == "full" else None})
                del ws
            del sets, y
            torch.cuda.empty_cache()
    return {"metric": "full and mean SS2D scans at every N=16 workload (us/call)",
            "unit": "us/call", "data": "synthetic",
            "timing": "HIP events on the launch stream around consecutive calls",
            "rows": rows}


def projections_bench(steps: int, warmup: int):
    """The selection projections of eq. 6 (vmb_ss2d_projections) at every
    N = 16 workload, in the scan's SEQ layout: the paper's broadcast timescale
    (R = 1, Linear_1) and VMamba's rank ceil(channels / 32). us per call with
    HIP events on the launch stream, enough input sets in turn that each call
    reads u from HBM; algorithmic bytes are u read plus delta, B and C
    written (the weights stay in cache), flops the two contractions."""
    import torch

    from paper_2412_16602_amd import vmb

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    g = torch.Generator(device=dev)
    g.manual_seed(3)
    rows = []
    for shp in (workloads.STAGE1, workloads.STAGE2, workloads.STAGE3, workloads.STAGE4,
                workloads.BATCHED_BF16, workloads.HIRES):
        b, K, Dc, L, N = shp.batch, 4, shp.channels, shp.L, shp.N
        dt = torch.bfloat16 if shp.dtype == "bf16" else torch.float32
        esz = 2 if shp.dtype == "bf16" else 4
        nbytes = b * K * L * (2 * Dc + 2 * N) * esz
        n_sets = max(1, min(8, -(-ROTATE_BYTES // nbytes)))
        us_in = [(torch.randn(b, K, Dc, L, device=dev, generator=g)).to(dt) for _ in range(n_sets)]
        delta = torch.empty(b, K, Dc, L, device=dev, dtype=dt)
        Bm = torch.empty(b, K, N, L, device=dev, dtype=dt)
        Cm = torch.empty_like(Bm)
        for R, bcast in ((1, True), (-(-Dc // 32), False)):
            W = torch.randn(K, R + 2 * N, Dc, device=dev, generator=g) / math.sqrt(Dc)
            Wdt = None if bcast else torch.randn(K, Dc, R, device=dev, generator=g) / math.sqrt(R)

            def call(i):
                vmb.vmb_ss2d_projections(us_in[i % n_sets], W, Wdt, delta, Bm, Cm, stream=stream)
            for i in range(warmup):
                call(i)
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            call(0)
            e1.record(stream)
            torch.cuda.synchronize()
            n = max(3, min(steps, int(0.2e6 / max(1.0, e0.elapsed_time(e1) * 1e3))))
            e0.record(stream)
            for i in range(n):
                call(i)
            e1.record(stream)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / n
            flops = 2 * b * K * L * Dc * ((R + 2 * N) + (0 if bcast else R))
            rows.append({"workload": shp.name, "dtype": shp.dtype, "R": R,
                         "timescale": "broadcast" if bcast else "low-rank", "us": round(us, 2),
                         "calls": n, "gbps": round(nbytes / (us * 1e-6) / 1e9, 1),
                         "hbm_frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                         "tflops": round(flops / (us * 1e-6) / 1e12, 2),
                         "mfma_f32_frac": round(flops / (us * 1e-6) / 1e12 / MFMA_F32_PEAK_TFLOPS,
                                                4)})
        del us_in, delta, Bm, Cm
        torch.cuda.empty_cache()
    return {"metric": "selection projections of eq. 6, every N=16 workload (us/call)",
            "unit": "us/call", "data": "synthetic",
            "timing": "HIP events on the launch stream around consecutive calls",
            "rows": rows}


def out_norm_bench(steps: int, warmup: int):
    """The channel normalisation and SiLU gate after the cross-merge
    (vmb_ss2d_out_norm) at every N = 16 workload's merged output
    [batch, channels, H*W]: us per call with HIP events on the launch stream,
    inputs rotated past the MALL; algorithmic bytes are y and z read and out
    written once."""
    import torch

    from paper_2412_16602_amd import vmb

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    g = torch.Generator(device=dev)
    g.manual_seed(4)
    rows = []
    for shp in (workloads.STAGE1, workloads.STAGE2, workloads.STAGE3, workloads.STAGE4,
                workloads.BATCHED_BF16, workloads.HIRES):
        b, Dc, P = shp.batch, shp.channels, shp.H * shp.W
        dt = torch.bfloat16 if shp.dtype == "bf16" else torch.float32
        esz = 2 if shp.dtype == "bf16" else 4
        nbytes = 3 * b * Dc * P * esz
        n_sets = max(1, min(8, -(-ROTATE_BYTES // nbytes)))
        sets = [(torch.randn(b, Dc, P, device=dev, generator=g).to(dt),
                 torch.randn(b, Dc, P, device=dev, generator=g).to(dt)) for _ in range(n_sets)]
        gamma = 1 + 0.1 * torch.randn(Dc, device=dev, generator=g)
        beta = 0.1 * torch.randn(Dc, device=dev, generator=g)
        out = torch.empty(b, Dc, P, device=dev, dtype=dt)

        def call(i):
            y, z = sets[i % n_sets]
            vmb.vmb_ss2d_out_norm(y, z, gamma, beta, 1e-5, out, stream=stream)
        for i in range(warmup):
            call(i)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        call(0)
        e1.record(stream)
        torch.cuda.synchronize()
        n = max(3, min(steps, int(0.2e6 / max(1.0, e0.elapsed_time(e1) * 1e3))))
        e0.record(stream)
        for i in range(n):
            call(i)
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / n
        rows.append({"workload": shp.name, "dtype": shp.dtype, "us": round(us, 2), "calls": n,
                     "gbps": round(nbytes / (us * 1e-6) / 1e9, 1),
                     "hbm_frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)})
        del sets, out
        torch.cuda.empty_cache()
    return {"metric": "channel LayerNorm + SiLU gate after the merge, every N=16 workload (us/call)",
            "unit": "us/call", "data": "synthetic",
            "timing": "HIP events on the launch stream around consecutive calls",
            "rows": rows}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--calibrate", action="store_true",
                    help="run a 256 MiB copy first (counter calibration dispatch)")
    ap.add_argument("--variants", action="store_true",
                    help="after the main line, print a line timing the mean scan's reading "
                         "variants (vmb_mean_scan_fwd_ex options) at the main workload")
    ap.add_argument("--workloads", action="store_true",
                    help="after the main line, print a line timing the full and mean scans "
                         "at every N=16 workload, both layouts")
    ap.add_argument("--projections", action="store_true",
                    help="after the main line, print a line timing the selection projections "
                         "of eq. 6 at every N=16 workload")
    ap.add_argument("--outnorm", action="store_true",
                    help="after the main line, print a line timing the channel LayerNorm and "
                         "SiLU gate after the merge at every N=16 workload")
    ap.add_argument("--table1", action="store_true",
                    help="after the main line, print a second JSON line: the one-state scan "
                         "on materialised inputs at the paper's Table 1 shapes")
    ap.add_argument("--table1-only", action="store_true",
                    help="print only the Table 1 line (for counter runs, which serialise "
                         "every dispatch)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this SS2D scan library runs on a single "
              "MI355X and has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    if args.calibrate:
        calibrate_copy()
    if args.table1_only:
        print(json.dumps(table1_bench(max(5, args.steps // 10), 3)), flush=True)
        return
    res, step_bytes, scan_bytes, n_rot, outputs = gpu_bench(args)
    full, mean = res["ss2d_full"], res["ss2d_mean"]
    sfull, smean = res["seq_full"], res["seq_mean"]
    kern_us = sfull["us"]
    achieved = scan_bytes / (kern_us * 1e-6) / 1e9
    shp = workloads.STAGE1
    elems = shp.batch * 4 * shp.channels * shp.N * shp.L
    achieved_tf = elems * FLOP_PER_ELEM / (kern_us * 1e-6) / 1e12
    hbm_frac = achieved / HBM_PEAK_GBPS
    alu_frac = achieved_tf / FP32_VECTOR_PEAK_TFLOPS
    rows = shp.batch * 4 * shp.channels * shp.L  # position-rows of one launch
    if hbm_frac >= alu_frac:
        bound = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                 "unit": "GB/s", "frac": round(hbm_frac, 4)}
        other = {"alu": {"achieved_tflops": round(achieved_tf, 3),
                         "peak_tflops": FP32_VECTOR_PEAK_TFLOPS, "frac": round(alu_frac, 4),
                         "flop_per_element": FLOP_PER_ELEM, "elements": elems}}
    else:
        bound = {"bound": "alu", "achieved": round(achieved_tf, 3),
                 "peak": FP32_VECTOR_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(alu_frac, 4)}
        other = {"hbm": {"achieved_gbps": round(achieved, 1), "peak_gbps": HBM_PEAK_GBPS,
                         "frac": round(hbm_frac, 4)}}
    step_prof = measured_step()
    step = {"us": round(full["us"], 3), "algorithmic_bytes": step_bytes,
            "hbm_frac": round(step_bytes / (full["us"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            "kernels": "full scan (2-D layout, per-direction outputs) + cross-merge",
            "kernels_us_traced": step_prof["kernels_us"] if step_prof else None,
            "traffic": step_prof["counter_bytes"] if step_prof else None}
    out = {
        "metric": METRIC,
        "value": round(full["us"], 3),
        "unit": "us/call",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(full["us"] / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": workloads.STAGE1.name, "batch": 1, "H": 56, "W": 56,
                   "channels": 192, "K": 4, "N": 16, "layout": "2d", "variant": "full",
                   "input_copies_rotated": n_rot},
        "gbps": round(step_bytes / (full["us"] * 1e-6) / 1e9, 1),
        "hbm_frac": round(step_bytes / (full["us"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
        "warm_us": round(full["warm_us"], 3),
        "per_call_us": full["dist"],
        "mean": {"us": round(mean["us"], 3), "warm_us": round(mean["warm_us"], 3),
                 "per_call_us": mean["dist"],
                 "gbps": round(step_bytes / (mean["us"] * 1e-6) / 1e9, 1),
                 "speedup_vs_full": round(full["us"] / mean["us"], 3)},
        "seq_scan": {"full_us": round(sfull["us"], 3), "mean_us": round(smean["us"], 3),
                     "bytes": scan_bytes,
                     "full_gbps": round(scan_bytes / (sfull["us"] * 1e-6) / 1e9, 1),
                     "mean_gbps": round(scan_bytes / (smean["us"] * 1e-6) / 1e9, 1),
                     "mean_speedup": round(sfull["us"] / smean["us"], 3)},
        "roofline": {**bound, "traffic": measured_traffic(),
                     "kernel": "full scan (positions over lanes), sequence layout",
                     "avg_us": round(kern_us, 3), "algorithmic_bytes": scan_bytes,
                     "bytes_per_position_row": round(scan_bytes / rows, 3),
                     "position_rows": rows, **other, "step": step},
    }
    if not args.no_cpu:
        out["cpu_baseline"], out["accuracy"] = cpu_baseline(args.cpu_budget, outputs)
    print(json.dumps(out), flush=True)
    if args.variants:
        print(json.dumps(variants_bench(args.steps, args.warmup)), flush=True)
    if args.workloads:
        print(json.dumps(workloads_bench(args.steps, 3)), flush=True)
    if args.projections:
        print(json.dumps(projections_bench(args.steps, 3)), flush=True)
    if args.outnorm:
        print(json.dumps(out_norm_bench(args.steps, 3)), flush=True)
    if args.table1:
        print(json.dumps(table1_bench(max(5, args.steps // 10), 3)), flush=True)


if __name__ == "__main__":
    main()
