"""The appendix-A searched plan on the GPU, for every network kind: the step
reports the search's exact peak, runs the plan's unit forwards, and gives the
no-checkpoint run's gradient bytes (recomputation reproduces activations
bit for bit whatever plan the search picks)."""
import pytest

import synth
from oracle import planner as PL, sizes as SZ

pytestmark = pytest.mark.gpu

CASES = {
    "mlp": dict(kind="mlp", depth=23, width=64, batch=16, seed=61),
    "resnet_basic": dict(kind="resnet_basic", blocks_per_stage=3, base=8, batch=4, image=16,
                         classes=10, seed=62),
    "lstm": dict(kind="lstm", T=21, batch=8, input=32, hidden=32, vocab=56, grad_chunk=4, seed=63),
    "resnet_bottleneck": dict(kind="resnet_bottleneck", stage_blocks=(3, 2), widths=(8, 16),
                              expansion=4, stem_channels=8, image=16, batch=2, classes=7, seed=64),
}


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("flags", [0, PL.FLAG_KEEP_LAST])
def test_searched_plan_identity(case, flags):
    import torch
    from paper_1604_06174_amd import ckpt as K
    from paper_1604_06174_amd.workload import GpuStep
    cfg = CASES[case]
    print(f"[search] case={case} flags={flags}", flush=True)
    d = synth.make(cfg)
    st = d["structure"]
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    plan, B, peak = step.net.search_plan(flags)
    b, a, q = SZ.tables(st)
    lb, cb = SZ.layer_and_cut_bytes(st)
    slot, extra = SZ.grad_layout(st, cfg.get("grad_chunk"))
    op, OB, opeak = PL.search(st.n, lb, cb, b, a, q, slot, extra, flags)
    assert (B, peak) == (OB, opeak) and plan.serialize() == op.serialize()
    loss, got_peak, stats = step.run(plan)
    torch.cuda.synchronize()
    assert got_peak == peak
    assert stats["unit_forwards"] == PL.unit_forwards(op)
    gbytes = step.grads_bytes()
    loss0, _, _ = step.run(step.plan(K.NONE))
    torch.cuda.synchronize()
    assert loss0 == loss
    assert step.grads_bytes() == gbytes
