"""Run a fixed number of checkpointed training steps for an external profiler.

    python -m paper_1604_06174_amd.profile_step --workload cifar110 --steps 2
    python -m paper_1604_06174_amd.profile_step --copy-mib 1024 --steps 3

The first form sets up one workload exactly as bench.py does (same seeded
inputs, same plan) and runs ``--steps`` steps on the current stream, with one
untimed step first so that one-time set-up does not show up in the per-kernel
counts of later steps.  The second form runs a plain device-to-device copy of
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
