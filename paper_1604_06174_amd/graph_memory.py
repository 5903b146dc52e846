"""Memory of each allocation strategy on a workload's node-granularity graph.

    python -m paper_1604_06174_amd.graph_memory [--workload cifar110]
    python -m paper_1604_06174_amd.graph_memory --workload mlp64 --run [--steps 20]
    python -m paper_1604_06174_amd.graph_memory --workload cifar110 --run

Builds the workload's forward graph at operator granularity, runs the
library's graph planner (Alg. 2 gradient-graph construction + section 3's
static allocator) for the paper's strategies -- no optimisation, in-place,
in-place + sharing, drop bn-relu (batch-norm and ReLU results mirrored), and a
segmented sublinear plan (every node mirrored except the outputs of every
s-th block, s = ceil(sqrt(blocks))) -- and prints one JSON line per strategy
with the planned bytes, the mirror nodes executed and the planning time.
With --run (nets whose library object provides the node graph: the residual
MLP and the CIFAR-shaped ResNet) each plan is also executed on the GPU by
train_step_graph -- synthetic inputs of the workload, a warm-up step, then
--steps timed steps between HIP events -- and the line gains ms/step, the
workspace bytes and, for comparison, the chain executor's ms/step and peak
bytes without checkpoints and under its sqrt plan.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def strategies(g):
    from synth import graphs as SG
    from paper_1604_06174_amd import ckpt as K
    nb = len(g["block_out"])
    s = math.isqrt(nb)
    s += 0 if s * s == nb else 1
    return [("no optimization", SG.mirror_none(g), K.ALLOC_NONE),
            ("inplace", SG.mirror_none(g), K.ALLOC_INPLACE),
            ("sharing", SG.mirror_none(g), K.ALLOC_SHARE),
            ("drop bn-relu", SG.mirror_bn_relu(g), K.ALLOC_SHARE),
            (f"sublinear, every {s} blocks kept", SG.mirror_segments(g, s), K.ALLOC_SHARE)]


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="cifar110")
    ap.add_argument("--run", action="store_true")
    ap.add_argument("--steps", type=int, default=20)
    args = ap.parse_args()
    import synth
    from synth import graphs as SG
    from paper_1604_06174_amd import ckpt as K
    cfg = synth.WORKLOADS[args.workload]
    g = SG.for_workload(cfg)
    step = timed = None
    if args.run:
        import torch
        from paper_1604_06174_amd.workload import GpuStep
        d = synth.make(cfg)
        step = GpuStep(cfg, d["params"], d["input"], d["target"])
        del d
        s = torch.cuda.current_stream()

        def timed(fn):
            fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(args.steps):
                fn()
            e1.record(s)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / args.steps

        chain = {}
        for cname, cplan in (("no_ckpt", step.plan(K.NONE)), ("sqrt", step.plan(K.SQRT))):
            ms = timed(lambda: step.run(cplan, stream=s, want_loss=False))
            _, peak, _ = step.run(cplan, stream=s, want_loss=False)
            chain[cname] = (round(ms, 4), round(peak / 1e9, 6))
    for name, mirror, strategy in strategies(g):
        t0 = time.perf_counter()
        plan = K.graph_plan(g["pred"], g["bytes"], g["flags"], mirror, strategy)
        dt = time.perf_counter() - t0
        info = plan.info()
        rec = {"workload": args.workload, "nodes": len(g["op"]), "strategy": name,
               "planned_gb": round(info["peak"] / 1e9, 6), "mirror_nodes": info["n_mirror"],
               "executed_nodes": info["n_exec"], "plan_ms": round(dt * 1e3, 3)}
        if args.run:
            gp = step.graph_plan(mirror, strategy)
            rec["ms_per_step"] = round(timed(lambda: step.run_graph(gp, stream=s, want_loss=False)), 4)
            rec["workspace_gb"] = round(step.net.graph_workspace_bytes(gp) / 1e9, 6)
            for cname, (ms, gb) in chain.items():
                rec[f"chain_{cname}_ms_per_step"] = ms
                rec[f"chain_{cname}_peak_gb"] = gb
        print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
