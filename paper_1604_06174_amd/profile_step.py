"""Run a fixed number of checkpointed training steps for an external profiler.

    python -m paper_1604_06174_amd.profile_step --workload cifar110 --steps 2
    python -m paper_1604_06174_amd.profile_step --workload resnet1000 --stage-blocks 3,3,3,3
    python -m paper_1604_06174_amd.profile_step --workload lstm4096 --seq-len 512
    python -m paper_1604_06174_amd.profile_step --copy-mib 1024 --steps 3

The first form sets up one workload exactly as bench.py does (same seeded
inputs, same plan) and runs ``--steps`` steps on the current stream, with one
untimed step first so that one-time set-up does not show up in the per-kernel
counts of later steps.  ``--stage-blocks`` gives a bottleneck net fewer blocks
per stage (the same layer widths, image and batch, so the same kernel instances
and launch shapes, in a shorter step); ``--seq-len`` does the same for the
LSTM (the same per-step launches over fewer steps).  The second form runs a plain device-to-device copy of
a known size, the reference that converts the HBM byte counters of a profiler
into bytes (a copy of S bytes reads S and writes S).
"""
from __future__ import annotations

import argparse
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="cifar110")
    ap.add_argument("--plan", default=None, choices=["sqrt", "greedy", "recursive", "search"])
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--copy-mib", type=int, default=0)
    ap.add_argument("--stage-blocks", default=None,
                    help="comma-separated blocks per stage (bottleneck nets only)")
    ap.add_argument("--seq-len", type=int, default=0, help="sequence length (LSTM only)")
    args = ap.parse_args()

    import torch

    if args.copy_mib > 0:
        n = args.copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"copied {n} bytes x {args.steps}", flush=True)
        return 0

    import synth
    from paper_1604_06174_amd import ckpt as K
    from paper_1604_06174_amd.workload import GpuStep

    cfg = dict(synth.WORKLOADS[args.workload])
    if args.plan:
        cfg["plan"] = args.plan
    if args.stage_blocks:
        if cfg["kind"] != "resnet_bottleneck":
            raise SystemExit("--stage-blocks applies to bottleneck nets only")
        cfg["stage_blocks"] = tuple(int(v) for v in args.stage_blocks.split(","))
    if args.seq_len:
        if cfg["kind"] != "lstm":
            raise SystemExit("--seq-len applies to the LSTM only")
        cfg["T"] = args.seq_len
    d = synth.make(cfg)
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    del d
    mode = cfg.get("plan", "sqrt")
    if mode == "search":
        plan, _, _ = step.net.search_plan()
    elif mode == "sqrt":
        plan = step.plan(K.SQRT, int(cfg.get("stride", 0)))
    elif mode == "greedy":
        lb, _ = step.net.layer_sizes()
        plan = step.plan(K.GREEDY, int(sum(lb) * cfg.get("budget_frac", 0.1)))
    else:
        plan = step.plan(K.RECURSIVE, 0)
    s = torch.cuda.current_stream()
    step.run(plan, stream=s, want_loss=False)
    torch.cuda.synchronize()
    print(f"{args.workload}: warm-up step done", flush=True)
    for k in range(args.steps):
        _, peak, stats = step.run(plan, stream=s, want_loss=False)
        torch.cuda.synchronize()
        print(f"{args.workload}: step {k + 1}/{args.steps} done, peak {peak} B, "
              f"{stats['kernel_launches']} launches", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
