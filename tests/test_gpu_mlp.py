"""GPU parity of the residual-MLP checkpointed step against the oracle.

For every plan mode the HIP step must give the oracle's loss and gradients
(float64 oracle; max |gpu - oracle| / max |oracle| per tensor <= 1e-4), the
same gradient bytes as the no-checkpoint run of the same kernels, the
oracle's peak-activation bytes and its unit-forward count.
"""
import numpy as np
import pytest

import synth
from oracle import nets, planner as PL, schedule as SCH, sizes as SZ

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _err(g, o):
    g = np.asarray(g, np.float64).reshape(-1)
    o = np.asarray(o, np.float64).reshape(-1)
    return float(np.max(np.abs(g - o)) / max(np.max(np.abs(o)), 1e-30))


def _oracle(d):
    chain = nets.Chain(d["structure"], d["params"])
    return nets.full_storage_step(chain, d["input"], d["target"])


def _modes(n, lb):
    out = [("none", PL.NONE, 0, None, 0), ("sqrt", PL.SQRT, 0, None, 0),
           ("sqrt_keep", PL.SQRT, 0, None, PL.FLAG_KEEP_LAST),
           ("greedy", PL.GREEDY, sum(lb) // 5, None, 0),
           ("recursive", PL.RECURSIVE, 0, None, 0),
           ("recursive_k3", PL.RECURSIVE, 3, None, 0)]
    if n > 3:
        out.append(("user", PL.USER, 0, [0, n // 2, n - 2], 0))
    return out


CASES = {
    # ragged: batch and width are not multiples of the 32/64 tiles
    "ragged": dict(kind="mlp", depth=9, width=72, batch=37, seed=51, w_var=1 / (72 * 9)),
    "tiles": dict(kind="mlp", depth=16, width=128, batch=64, seed=52),
    "cfg_mlp64": synth.WORKLOADS["mlp64"],
}


@pytest.mark.parametrize("case", list(CASES))
def test_mlp_step_parity_all_modes(case):
    import torch
    from paper_1604_06174_amd.workload import GpuStep
    cfg = CASES[case]
    print(f"[mlp parity] case={case} cfg={cfg}", flush=True)
    d = synth.make(cfg)
    loss_o, grads_o = _oracle(d)
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    st = d["structure"]
    b, a, q = SZ.tables(st)
    lb, cb = SZ.layer_and_cut_bytes(st)
    ref_bytes = None
    for name, mode, budget, user, flags in _modes(st.n, lb):
        plan = step.plan(mode, budget, user, flags)
        step.grads.fill_(float("nan"))
        loss, peak, stats = step.run(plan)
        torch.cuda.synchronize()
        op = PL.plan(st.n, lb, cb, budget, mode, user, flags)
        assert peak == PL.account(op, b, a, q).peak, name
        assert stats["unit_forwards"] == PL.unit_forwards(op), name
        assert stats["unit_backwards"] == st.n
        assert abs(loss - loss_o) <= TOL * abs(loss_o), (name, loss, loss_o)
        g = step.grads_host()
        for k, v in grads_o.items():
            e = _err(g[k], v)
            assert e <= TOL, (name, k, e)
        gb = step.grads_bytes()
        if ref_bytes is None:
            ref_bytes = gb
        assert gb == ref_bytes, f"{name}: gradients differ from the no-checkpoint run"
    # determinism: a second run of the same plan reproduces the bytes
    step.run(step.plan(PL.SQRT))
    torch.cuda.synchronize()
    assert step.grads_bytes() == ref_bytes


def test_mlp_loss_dev_and_stream():
    import torch
    from paper_1604_06174_amd.workload import GpuStep
    cfg = CASES["tiles"]
    d = synth.make(cfg)
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    s = torch.cuda.Stream()
    plan = step.plan(PL.SQRT)
    loss, _, _ = step.run(plan, stream=s, want_loss=False)
    assert loss is None
    s.synchronize()
    loss_o, _ = _oracle(d)
    assert abs(step.loss_dev.item() - loss_o) <= TOL * abs(loss_o)
