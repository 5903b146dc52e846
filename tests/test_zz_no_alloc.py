"""train_step_static (the training step on the library's static per-GPU
scratch, for callers that cannot allocate) against train_step on a caller
workspace: loss and every gradient bit for bit, on two calls in a row, the
second with a smaller input (so the first call's leftovers sit in the
scratch), then a third on the first net again."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

CASES = [
    # the CIFAR-shaped basic-block net (batch-norm partial sums in the
    # operator region of the scratch), then the residual MLP, smaller
    dict(kind="resnet_basic", blocks_per_stage=2, base=8, batch=16, image=16, classes=10, seed=71),
    dict(kind="mlp", depth=9, width=72, batch=37, seed=72, w_var=1 / (72 * 9)),
]


def _pair(cfg, plan_mode):
    import torch
    from paper_1604_06174_amd import ckpt as K
    from paper_1604_06174_amd.workload import GpuStep
    d = synth.make(cfg)
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    plan = step.plan(plan_mode)
    need = step.net.workspace_bytes(plan)
    assert need <= K.STATIC_SCRATCH_BYTES
    # the step writes every gradient tensor but not the padding between them:
    # both runs start from the same fill
    step.grads.fill_(float("nan"))
    loss_ref, peak_ref, st_ref = step.run(plan)
    torch.cuda.synchronize()
    ref = step.grads_bytes()
    step.grads.fill_(float("nan"))
    s = torch.cuda.current_stream()
    loss, peak, st = K.train_step_static(step.net, step.params, step.grads, step.input, step.target,
                                         plan, s, step.loss_dev)
    torch.cuda.synchronize()
    print(f"  {cfg['kind']}: workspace {need} B, loss {loss:.7f} (train_step {loss_ref:.7f})",
          flush=True)
    assert loss == loss_ref
    assert peak == peak_ref
    assert st == st_ref
    assert step.grads_bytes() == ref
    assert float(step.loss_dev.item()) == loss_ref
    return need


def test_static_scratch_matches_train_step():
    from paper_1604_06174_amd import ckpt as K
    print("[no-alloc] train_step_static vs train_step", flush=True)
    n0 = _pair(CASES[0], K.SQRT)
    n1 = _pair(CASES[1], K.SQRT)
    assert n1 < n0
    _pair(CASES[0], K.RECURSIVE)
