"""Memory of each allocation strategy on a workload's node-granularity graph.

    python -m paper_1604_06174_amd.graph_memory [--workload cifar110]

Builds the workload's forward graph at operator granularity, runs the
library's graph planner (Alg. 2 gradient-graph construction + section 3's
static allocator) for the paper's strategies -- no optimisation, in-place,
in-place + sharing, drop bn-relu (batch-norm and ReLU results mirrored), and a
segmented sublinear plan (every node mirrored except the outputs of every
s-th block, s = ceil(sqrt(blocks))) -- and prints one JSON line per strategy
with the planned bytes, the mirror nodes executed and the planning time.
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
    args = ap.parse_args()
    import synth
    from synth import graphs as SG
    from paper_1604_06174_amd import ckpt as K
    cfg = synth.WORKLOADS[args.workload]
    g = SG.for_workload(cfg)
    for name, mirror, strategy in strategies(g):
        t0 = time.perf_counter()
        plan = K.graph_plan(g["pred"], g["bytes"], g["flags"], mirror, strategy)
        dt = time.perf_counter() - t0
        info = plan.info()
        print(json.dumps({"workload": args.workload, "nodes": len(g["op"]), "strategy": name,
                          "planned_gb": round(info["peak"] / 1e9, 6),
                          "mirror_nodes": info["n_mirror"], "executed_nodes": info["n_exec"],
                          "plan_ms": round(dt * 1e3, 3)}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
