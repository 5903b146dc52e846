"""GPU: a training step recorded as a HIP graph (step_graph_create) and
replayed (step_graph_launch) gives the gradients and the loss of the same step
submitted launch by launch, bit for bit, for every network kind and a
one-level and a recursive plan.

Each recorded step is replayed three times with other work in between (a step
under another plan, gradient buffers overwritten with NaN, host
synchronisation), and every replay is checked; a replay after the parameters
were changed in place must give the step of the new parameters (the recording
keeps addresses, not values).  A fourth network, the full-size CIFAR-shaped
ResNet-110, is recorded under the sqrt plan the benchmark times.
"""
import numpy as np
import pytest

import synth
from paper_1604_06174_amd import ckpt as K

pytestmark = pytest.mark.gpu

CASES = {
    "mlp": dict(kind="mlp", depth=9, width=72, batch=37, seed=81, w_var=1 / (72 * 9)),
    "resnet": dict(kind="resnet_basic", blocks_per_stage=2, base=16, batch=8, image=16, classes=10,
                   seed=82),
    "resnet_drop": dict(kind="resnet_basic", blocks_per_stage=2, base=16, batch=8, image=16,
                        classes=10, seed=83, drop_bn_relu=1),
    "lstm": dict(kind="lstm", T=20, batch=16, input=64, hidden=64, vocab=200, grad_chunk=8, seed=84),
    "bottleneck": dict(kind="resnet_bottleneck", stage_blocks=(2, 2), widths=(8, 16), expansion=4,
                       stem_channels=8, image=16, batch=2, classes=7, seed=85),
    "cifar110": synth.WORKLOADS["cifar110"],
}


def _eager(step, plan):
    import torch
    step.grads.fill_(float("nan"))
    step.run(plan, want_loss=False)
    torch.cuda.synchronize()
    return step.grads.cpu().numpy().tobytes(), step.loss_dev.cpu().numpy().tobytes()


@pytest.mark.parametrize("case", list(CASES))
def test_recorded_step_replays_bit_identical(case):
    import torch
    from paper_1604_06174_amd.workload import GpuStep
    cfg = CASES[case]
    print(f"[step graph] case={case}", flush=True)
    d = synth.make(cfg)
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    plans = {"sqrt": step.plan(K.SQRT)}
    if case != "cifar110":
        plans["recursive"] = step.plan(K.RECURSIVE)
    other = step.plan(K.NONE)
    step.workspace(other)
    s = torch.cuda.Stream()
    for pname, plan in plans.items():
        tag = f"{case}/{pname}"
        ref = _eager(step, plan)
        g = step.record(plan, s)
        assert g.stats["unit_forwards"] >= step.net.n, tag
        for r in range(3):
            _eager(step, other)                # other work between the replays
            step.grads.fill_(float("nan"))
            step.loss_dev.fill_(float("nan"))
            torch.cuda.synchronize()
            g.launch(s)
            torch.cuda.synchronize()
            got = (step.grads.cpu().numpy().tobytes(), step.loss_dev.cpu().numpy().tobytes())
            assert got[1] == ref[1], f"{tag} replay {r}: loss"
            assert got[0] == ref[0], f"{tag} replay {r}: gradients"
        # the recording reads the parameters' current contents
        saved = step.params.clone()
        step.params.mul_(0.5)
        ref2 = _eager(step, plan)
        assert ref2 != ref, tag
        step.grads.fill_(float("nan"))
        torch.cuda.synchronize()
        g.launch(s)
        torch.cuda.synchronize()
        assert step.grads.cpu().numpy().tobytes() == ref2[0], f"{tag}: after a parameter change"
        step.params.copy_(saved)
        g.close()
        torch.cuda.synchronize()


def test_record_rejects_default_stream_and_timing():
    import torch
    from paper_1604_06174_amd.workload import GpuStep
    cfg = CASES["mlp"]
    d = synth.make(cfg)
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    plan = step.plan(K.SQRT)
    ws = step.workspace(plan)
    with pytest.raises(K.CkptError) as e:
        K.step_graph_create(step.net, step.params, step.grads, step.input, step.target, plan, ws,
                            ws.numel(), 0, step.loss_dev)
    assert e.value.code == K.E_INVALID
    s = torch.cuda.Stream()
    step.net.timing_enable(True)
    try:
        with pytest.raises(K.CkptError) as e:
            step.record(plan, s)
        assert e.value.code == K.E_INVALID
    finally:
        step.net.timing_enable(False)
    # the stream is usable afterwards: recording still works
    g = step.record(plan, s)
    g.launch(s)
    torch.cuda.synchronize()
    assert np.isfinite(step.loss_dev.item())
