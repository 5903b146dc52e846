#!/usr/bin/env python3
"""Benchmark of the checkpointed training step on one MI355X.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload resnet1000]

Default workload: the ImageNet-shaped ~1000-layer bottleneck ResNet of section
5.2 (stem + 333 bottleneck blocks split 32/64/205/32, 224x224 input, batch 32,
bf16 activations, fp32 batch-norm statistics) with the budget-driven greedy
plan of Alg. 3 at a budget of 10% of the full-storage activation bytes.  A
step is one whole checkpointed train step: forward keeping only segment
boundaries, loss head, and for every segment in reverse its forward re-run
followed by its backward, producing every gradient.  Inputs are seeded
synthetic tensors already resident in HBM.

Printed (one JSON line): samples/s of the checkpointed step (mean over the
timed steps; the median of the per-step times is given too), its peak
activation bytes (exact, from the static layout) next to the bytes the step
measurably wrote in each workspace region, the recompute overhead (step time /
the same kernels without checkpointing), the dominant kernel's roofline
position from HIP events that its launches stamp with the kernels' own start
and end, in a second timed pass (against MFMA peak when the family's
arithmetic intensity is at or above the ridge point, else against HBM
bandwidth; both fractions are given), and the CPU oracle's full-storage step
(float32 NumPy) on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "checkpointed train-step samples/s + peak activation GB + recompute overhead ×"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
HBM_GBS = 8000.0


def _plan_args(cfg, net):
    from paper_1604_06174_amd import ckpt as K
    lb, _ = net.layer_sizes()
    mode = cfg.get("plan", "sqrt")
    if mode == "search":
        return "search", None, "search"
    if mode == "sqrt":
        return K.SQRT, int(cfg.get("stride", 0)), "sqrt"
    if mode == "greedy":
        return K.GREEDY, int(sum(lb) * cfg.get("budget_frac", 0.1)), "greedy"
    if mode == "recursive":
        return K.RECURSIVE, int(cfg.get("fanout", 1)), "recursive"
    raise ValueError(mode)


def _traffic(workload):
    """Measured HBM bytes per launch of the dominant kernel family, from the
    calibrated rocprofv3 FETCH_SIZE / WRITE_SIZE runs recorded in
    profiles/traffic.json; None when none was recorded for this workload or
    when a source file the counters were taken on has changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)["workloads"][workload]
        h = hashlib.sha256()
        for src in rec["sources"]:
            with open(os.path.join(ROOT, src), "rb") as f:
                h.update(f.read())
    except (OSError, KeyError, ValueError):
        return None
    if h.hexdigest() != rec["sources_sha256"]:
        return None
    return rec


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _cpu_baseline(cfg, sample_batch, d_full):
    """The oracle's plain full-storage training step (float32 NumPy, no bf16
    rounding) of the same network on a smaller batch (the same parameters, the
    first samples of the batch; for the LSTM a prefix of the time steps);
    samples/s = sample / wall time, scaled to the full step."""
    import numpy as np
    import synth
    from oracle import nets, units as U
    try:
        from threadpoolctl import threadpool_info
        threads = max([t.get("num_threads", 1) for t in threadpool_info()
                       if t.get("internal_api") in ("openblas", "mkl", "blis")] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    c = dict(cfg)
    scale = 1.0
    if cfg["kind"] == "lstm":
        # a prefix of the sequences: the work grows linearly with the steps
        c["T"] = sample_batch
        scale = sample_batch / cfg["T"]
        what = f"{sample_batch} of its {cfg['T']} time steps (all {cfg['batch']} sequences)"
        n_samples = cfg["batch"]
    else:
        c["batch"] = sample_batch
        what = f"{sample_batch} of its {cfg['batch']} samples"
        n_samples = sample_batch
    structure = synth.structure(c)
    inp, tgt = d_full["input"][:sample_batch], d_full["target"][:sample_batch]
    chain = nets.Chain(structure, d_full["params"], U.Prec(np.float32, False))
    t0 = time.perf_counter()
    nets.full_storage_step(chain, inp, tgt)
    dt = time.perf_counter() - t0
    return {"value": n_samples * scale / dt, "unit": "samples/s", "cores": int(threads),
            "kind": "oracle", "dtype": "f32", "cpu_model": _cpu_model(),
            "sample": f"one float32 NumPy full-storage step of the same network on "
                      f"{what}, scaled to the full step; {dt:.1f} s wall"}


def _touched(ws, lo, hi, chunk=1 << 20):
    """Bytes from `lo` up to the last byte in [lo, hi) that differs from the
    0xFF fill (0 when none does); every value the step stores is finite, so an
    all-ones bf16 / fp32 word marks memory it never wrote."""
    import torch
    if hi <= lo:
        return 0
    v = ws[lo:hi]
    n = v.numel()
    full = n // chunk
    last = -1
    if n > full * chunk:
        tail = (v[full * chunk:] != 255).nonzero()
        if tail.numel():
            last = full * chunk + int(tail[-1])
    if last < 0 and full:
        hit = (v[:full * chunk].view(full, chunk) != 255).any(dim=1).nonzero()
        if hit.numel():
            c = int(hit[-1])
            last = c * chunk + int((v[c * chunk:(c + 1) * chunk] != 255).nonzero()[-1])
    return last + 1


def _measured_regions(step, plan, acc, stream):
    """One more step on a workspace filled with 0xFF: per region (kept
    boundaries, re-run arena, gradient buffers), the extent the step wrote."""
    import torch
    al = lambda x: (x + 255) // 256 * 256
    ws = step.workspace(plan)
    ws.fill_(255)
    torch.cuda.synchronize()
    step.run(plan, stream=stream, want_loss=False)
    torch.cuda.synchronize()
    o_ck, o_ar, o_gr = 0, al(acc["ckpt"]), al(acc["ckpt"]) + al(acc["arena"])
    out = {"ckpt": _touched(ws, o_ck, o_ck + acc["ckpt"]),
           "arena": _touched(ws, o_ar, o_ar + acc["arena"]),
           "grad": _touched(ws, o_gr, o_gr + acc["grad"])}
    out["total"] = sum(out.values())
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="resnet1000")
    ap.add_argument("--plan", default=None, choices=["sqrt", "greedy", "recursive", "search"],
                    help="override the workload's plan (search: the appendix-A budget search)")
    ap.add_argument("--fanout", type=int, default=0,
                    help="recursive plan: boundaries stored per level (section 4.4's k; default 1)")
    ap.add_argument("--drop-bn-relu", action="store_true",
                    help="residual CNNs: keep only convolution outputs and re-form batch norm + "
                         "ReLU from them when read")
    ap.add_argument("--graph", action="store_true",
                    help="also time each step recorded once as a HIP graph and replayed "
                         "(step_graph_create / step_graph_launch)")
    ap.add_argument("--cpu-sample", type=int, default=-1,
                    help="batch (LSTM: time steps) of the CPU oracle sample; 0 skips it, -1 picks "
                         "about 10-30 s of oracle work for the workload")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the checkpointed step is "
                                   "measured per device; multi-GPU sharding is not built",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch
    import synth
    from paper_1604_06174_amd import ckpt as K
    from paper_1604_06174_amd.workload import GpuStep

    cfg = dict(synth.WORKLOADS[args.workload])
    if args.drop_bn_relu:
        if cfg["kind"] not in ("resnet_basic", "resnet_bottleneck"):
            print(json.dumps({"error": "--drop-bn-relu applies to the residual CNNs"}))
            sys.exit(2)
        cfg["drop_bn_relu"] = 1
    d = synth.make(cfg)
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    if args.plan:
        cfg["plan"] = args.plan
    if args.fanout:
        if cfg.get("plan") != "recursive":
            print(json.dumps({"error": "--fanout applies to the recursive plan"}))
            sys.exit(2)
        cfg["fanout"] = args.fanout
    mode, budget, mode_name = _plan_args(cfg, step.net)
    if mode == "search":
        plan, budget, _ = step.net.search_plan()
    else:
        plan = step.plan(mode, budget)
    none = step.plan(K.NONE)
    acc = step.net.accounting(plan)
    acc_none = step.net.accounting(none)
    step.workspace(none)  # the larger workspace serves both plans
    s = torch.cuda.Stream()  # a created stream (default priority): steps can be recorded on it

    def run(p, k):
        st = None
        for _ in range(k):
            _, _, st = step.run(p, stream=s, want_loss=False)
        return st

    stats = run(plan, args.warmup)
    run(none, args.warmup)
    torch.cuda.synchronize()

    def timed(launch, per_step=None):
        # events on the stream the steps run on: one pair around all K steps
        # (the mean), and one per step (the median)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        torch.cuda.synchronize()
        ev[0].record(s)
        for k in range(args.steps):
            launch()
            ev[k + 1].record(s)
        torch.cuda.synchronize()
        if per_step is not None:
            per_step.extend(ev[k].elapsed_time(ev[k + 1]) for k in range(args.steps))
        return ev[0].elapsed_time(ev[-1]) / args.steps

    step_ms = []
    ms = timed(lambda: step.run(plan, stream=s, want_loss=False), step_ms)
    ms_none = timed(lambda: step.run(none, stream=s, want_loss=False))
    ms_median = float(np.median(step_ms))
    graph_ms = None
    if args.graph:  # each step recorded once as a HIP graph, then replayed
        graphs = {"plan": step.record(plan, s), "none": step.record(none, s)}
        for g in graphs.values():
            for _ in range(args.warmup):
                g.launch(s)
        torch.cuda.synchronize()
        graph_ms = {"ms_per_step": round(timed(lambda: graphs["plan"].launch(s)), 4),
                    "ms_per_step_no_ckpt": round(timed(lambda: graphs["none"].launch(s)), 4)}
    loss = float(step.loss_dev.item())
    # bytes the checkpointed step writes in each region of the workspace,
    # next to the planned (exact) peak; then the device allocator's
    # high-water mark of the whole process (parameters, gradients, batch,
    # workspace for the no-checkpoint plan, which is the larger)
    written = _measured_regions(step, plan, acc, s)
    device_hwm = torch.cuda.max_memory_allocated()

    # second timed pass: every launch of the dominant kernel family stamps an
    # event pair with its own start and end
    step.net.timing_enable(True)
    run(plan, args.steps)
    torch.cuda.synchronize()
    kt = step.net.timing_read()
    kr = step.net.timing_roofline(PEAK_TFLOPS[cfg.get("dtype", "f32")] * 1e12, HBM_GBS * 1e9)
    step.net.timing_enable(False)

    dtype = cfg.get("dtype", "f32")  # "bf16": bf16 GEMM operands, fp32 accumulation
    tflops = kt["flops"] / (kt["ms"] / 1e3) / 1e12 if kt["ms"] > 0 else 0.0
    gbs = kt["bytes"] / (kt["ms"] / 1e3) / 1e9 if kt["ms"] > 0 else 0.0
    peak_f = PEAK_TFLOPS[dtype]
    # roofline placement: below the ridge (peak flops / peak bandwidth) the
    # family's arithmetic intensity bounds it by HBM, above it by MFMA
    ai = kt["flops"] / kt["bytes"] if kt["bytes"] > 0 else float("inf")
    ridge = peak_f * 1e12 / (HBM_GBS * 1e9)
    if ai >= ridge:
        bound, achieved, peak, unit = "mfma", tflops, peak_f, "TFLOP/s"
    else:
        bound, achieved, peak, unit = "hbm", gbs, HBM_GBS, "GB/s"
    # counters were taken on the workload's default layout and plan family only
    tr = None if args.drop_bn_relu else _traffic(args.workload)
    alg_bytes = kt["bytes"] / max(kt["launches"], 1)
    roof = {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4),
            "arithmetic_intensity": round(ai, 2), "ridge": round(ridge, 2),
            "frac_mfma": round(tflops / peak_f, 4), "frac_hbm": round(gbs / HBM_GBS, 4),
            "traffic": tr["traffic_bytes_per_launch"] if tr else None,
            "algorithmic_bytes_per_launch": round(alg_bytes),
            "traffic_over_algorithmic": round(tr["traffic_bytes_per_launch"] / alg_bytes, 3) if tr else None,
            "kernel": kt["kernel"], "launches": kt["launches"],
            "avg_launch_us": round(kt["ms"] * 1e3 / max(kt["launches"], 1), 3),
            "flops_per_launch": kt["flops"] / max(kt["launches"], 1),
            "tflops_algorithmic": round(tflops, 3), "hbm_gbs_algorithmic": round(gbs, 1),
            # every launch against its own bound: sum of max(flops / peak, bytes / 8 TB/s)
            # over the family's launches, over their measured time
            "frac_of_roofline_time": round(kr["roofline_ms"] / kr["kernel_ms"], 4) if kr["kernel_ms"] > 0 else None,
            # launches of the family on two streams overlap (the bottleneck net's
            # weight gradients): the time at least one of them ran, per step, and
            # the family's rate over that time at the same bound
            "busy_ms_per_step": round(kr["busy_ms"] / args.steps, 3),
            "summed_ms_per_step": round(kr["kernel_ms"] / args.steps, 3),
            "frac_over_busy_time": round((kt["flops"] if bound == "mfma" else kt["bytes"]) /
                                         (kr["busy_ms"] / 1e3) / (peak * (1e12 if bound == "mfma" else 1e9)), 4)
            if kr["busy_ms"] > 0 else None}

    cpu = None
    sample = args.cpu_sample
    if sample < 0:
        sample = {"lstm": 16, "resnet_bottleneck": 1, "resnet_basic": 32}.get(cfg["kind"], 128)
    if sample > 0:
        if cfg["kind"] == "lstm":
            cpu = _cpu_baseline(cfg, min(sample, cfg["T"]), d)
        else:
            cpu = _cpu_baseline(cfg, min(sample, cfg["batch"]), d)

    batch = cfg["batch"]
    out = {
        "metric": METRIC,
        "value": round(batch / (ms / 1e3), 3),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "ms_per_step_median": round(ms_median, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": args.workload + ("+drop_bn_relu" if args.drop_bn_relu else ""),
                   "kind": cfg["kind"], "batch": batch,
                   "units": step.net.n, "plan": mode_name,
                   "stride_or_budget": budget, "cuts": len(plan.cuts()),
                   **({"fanout": budget} if mode_name == "recursive" else {})},
        "peak_activation_gb": round(acc["peak"] / 1e9, 6),
        "peak_activation_gb_no_ckpt": round(acc_none["peak"] / 1e9, 6),
        "peak_activation_gb_written": round(written["total"] / 1e9, 6),
        "peak_regions_bytes": {"planned": {k: acc[k] for k in ("ckpt", "arena", "grad")},
                               "written": {k: written[k] for k in ("ckpt", "arena", "grad")}},
        "device_allocated_hwm_gb": round(device_hwm / 1e9, 6),
        "recompute_overhead_x": round(ms / ms_none, 4),
        "ms_per_step_no_ckpt": round(ms_none, 4),
        **({"hip_graph_replay": graph_ms} if graph_ms else {}),
        "unit_forwards_per_step": stats["unit_forwards"],
        "kernel_launches_per_step": stats["kernel_launches"],
        "loss": loss,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
