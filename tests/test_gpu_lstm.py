"""GPU parity of the LSTM checkpointed step (bf16 GEMM operands, fp32
accumulation and cell state) against the oracle.

Two bars per gradient tensor (max |gpu - oracle| / max |oracle|):
* 2e-2 against the float64 oracle without rounding (the bf16 bar);
* 2e-3 against the oracle that rounds to bf16 at the same points as the GPU
  (weights once per step, x_t, h_t, and the dz / softmax-gradient GEMM
  operands): a float32 run of that oracle stays within 1.6e-4 of its float64
  run on these shapes, so 2e-3 leaves room for the rare bf16 rounding flips.
Every plan must also give the no-checkpoint run's gradient bytes (the weight
gradients accumulate over fixed chunks of steps in backward order whatever the
plan), the oracle's peak bytes and its unit-forward count.
"""
import numpy as np
import pytest

import synth
from oracle import nets, planner as PL, sizes as SZ, units as U

pytestmark = pytest.mark.gpu


def _err(g, o):
    g = np.asarray(g, np.float64).reshape(-1)
    o = np.asarray(o, np.float64).reshape(-1)
    return float(np.max(np.abs(g - o)) / max(np.max(np.abs(o)), 1e-30))


CASES = {
    "tiny": dict(kind="lstm", T=9, batch=3, input=16, hidden=24, vocab=40, grad_chunk=4, seed=71),
    "mid": dict(kind="lstm", T=20, batch=16, input=64, hidden=64, vocab=200, grad_chunk=8, seed=72),
    "wide": dict(kind="lstm", T=6, batch=64, input=128, hidden=128, vocab=1000, seed=73),
}


@pytest.mark.parametrize("case", list(CASES))
def test_lstm_step_parity_all_modes(case):
    import torch
    from paper_1604_06174_amd.workload import GpuStep
    cfg = CASES[case]
    print(f"[lstm parity] case={case} cfg={cfg}", flush=True)
    d = synth.make(cfg)
    loss64, g64 = nets.full_storage_step(nets.Chain(d["structure"], d["params"]), d["input"], d["target"])
    lossb, gb = nets.full_storage_step(nets.Chain(d["structure"], d["params"], U.Prec(np.float64, True)),
                                       d["input"], d["target"])
    step = GpuStep(cfg, d["params"], d["input"], d["target"])
    st = d["structure"]
    b, a, q = SZ.tables(st)
    slot, extra = SZ.grad_layout(st, cfg.get("grad_chunk"))
    lb, cb = SZ.layer_and_cut_bytes(st)
    n = st.n
    modes = [("none", PL.NONE, 0, None, 0), ("sqrt", PL.SQRT, 0, None, 0),
             ("stride2_keep", PL.SQRT, 2, None, PL.FLAG_KEEP_LAST),
             ("greedy", PL.GREEDY, sum(lb) // 3, None, 0), ("recursive", PL.RECURSIVE, 0, None, 0),
             ("recursive_k3", PL.RECURSIVE, 3, None, 0),
             ("user", PL.USER, 0, [0, n - 2], 0)]
    ref = None
    for name, mode, budget, user, flags in modes:
        plan = step.plan(mode, budget, user, flags)
        step.grads.fill_(float("nan"))
        loss, peak, stats = step.run(plan)
        torch.cuda.synchronize()
        op = PL.plan(n, lb, cb, budget, mode, user, flags)
        assert peak == PL.account(op, b, a, q, slot, extra).peak, name
        assert stats["unit_forwards"] == PL.unit_forwards(op), name
        assert abs(loss - lossb) <= 2e-3 * abs(lossb), (name, loss, lossb)
        g = step.grads_host()
        worst_b = max((_err(g[k], v), k) for k, v in gb.items())
        worst_64 = max((_err(g[k], v), k) for k, v in g64.items())
        assert worst_b[0] <= 2e-3, (name, worst_b)
        assert worst_64[0] <= 2e-2, (name, worst_64)
        gbytes = step.grads_bytes()
        if ref is None:
            ref = gbytes
        assert gbytes == ref, f"{name}: gradients differ from the no-checkpoint run"
