"""GPU: training steps over the residual MLP's operator-level graph, planned by
Alg. 2 (mirror nodes) and the section-3 allocator.

For every mirror plan (none; ReLU results dropped; segments of 1 and 3 blocks
kept; everything mirrored twice) and every allocation strategy (no
optimisation, in-place, in-place + sharing): the gradients and the loss are
bit-identical to the chain executor's no-checkpoint step (whose parity with the
oracle the MLP tests establish; the node operators perform the same float
operations in the same order), the planned bytes equal the oracle planner's,
and the numbers of forward, mirror and gradient nodes run equal the plan's.
"""
import pytest

import synth
from oracle import graph as OG
from paper_1604_06174_amd import ckpt as K
from synth import graphs as SG

pytestmark = pytest.mark.gpu

CASES = {
    "ragged": dict(kind="mlp", depth=9, width=72, batch=37, seed=51, w_var=1 / (72 * 9)),
    "tiles": dict(kind="mlp", depth=16, width=128, batch=64, seed=52),
    "cfg_mlp64": synth.WORKLOADS["mlp64"],
}


def _mirrors(g):
    n = len(g["op"])
    twice = [0 if (not g["pred"][v] or g["op"][v] == "loss") else 2 for v in range(n)]
    return {"none": SG.mirror_none(g), "relu": SG.mirror_bn_relu(g),
            "seg1": SG.mirror_segments(g, 1), "seg3": SG.mirror_segments(g, 3), "twice": twice}


@pytest.mark.parametrize("case", list(CASES))
def test_graph_steps_match_chain_step(case):
    import torch
    from paper_1604_06174_amd.workload import GpuStep
    cfg = CASES[case]
    print(f"[graph step] case={case} cfg={cfg}", flush=True)
    d = synth.make(cfg)
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    loss_ref, _, _ = step.run(step.plan(K.NONE))
    torch.cuda.synchronize()
    ref_t = step.grads_host()
    sg = SG.mlp(cfg["depth"], cfg["width"], cfg["batch"])
    for mname, mirror in _mirrors(sg).items():
        for strategy in (K.ALLOC_NONE, K.ALLOC_INPLACE, K.ALLOC_SHARE):
            plan = step.graph_plan(mirror, strategy)
            op = OG.plan(sg["pred"], sg["bytes"], sg["flags"], mirror, strategy)
            step.grads.fill_(float("nan"))
            loss, peak, stats = step.run_graph(plan)
            torch.cuda.synchronize()
            tag = f"{case}/{mname}/{strategy}"
            assert peak == op.peak, tag
            kinds = [op.nodes[w].kind for w in op.order]
            assert stats["unit_forwards"] == kinds.count(OG.FWD) + kinds.count(OG.MIRROR), tag
            assert stats["unit_backwards"] == kinds.count(OG.GRAD), tag
            assert loss == loss_ref, tag
            got = step.grads_host()
            bad = [k for k in ref_t if got[k].tobytes() != ref_t[k].tobytes()]
            assert not bad, f"{tag}: gradients differ from the chain step: {bad[:8]}"
        print(f"  {mname}: planned {op.peak} B (sharing), {op.n_mirror} mirrors", flush=True)
