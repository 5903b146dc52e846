"""Pins of the oracle's checkpointed executors (CPU only).

* The Alg. 1 executor (every one-level plan, with and without keeping the
  last segment) and the recursive executor return gradients bit-identical to
  the full-storage step: recomputation reproduces the dropped activations
  exactly, so the weight gradient is the same (section 5.1).
* Their unit-forward counters equal the planner's counts: 2n for a literal
  one-level plan, n + n(log2 n + 1)/2 for the recursive plan at powers of two,
  and the recursive executor keeps at most ceil(log2 n) boundaries at once.
"""
import math

import numpy as np
import pytest

import synth
from oracle import nets, planner as PL, schedule as SCH, sizes as SZ

TINY = {
    "mlp": dict(kind="mlp", depth=8, width=8, batch=3, seed=31, w_var=0.1),
    "cnn": dict(kind="resnet_basic", blocks_per_stage=2, base=2, batch=2, image=8, classes=3, seed=32),
    "lstm": dict(kind="lstm", T=9, batch=2, input=3, hidden=4, vocab=5, seed=33),
    "bottleneck": dict(kind="resnet_bottleneck", stage_blocks=(2, 1), widths=(2, 3), expansion=2,
                       stem_channels=4, batch=2, image=16, classes=3, seed=34),
}


def _same(ga, gb):
    assert ga.keys() == gb.keys()
    for k in ga:
        assert np.array_equal(ga[k], gb[k]), k


def _plans(n):
    lb, cb = [1] * n, [1] * (n - 1) + [0]
    out = [PL.plan(n, lb, cb, 0, PL.SQRT), PL.plan(n, lb, cb, 0, PL.SQRT, flags=PL.FLAG_KEEP_LAST),
           PL.plan(n, lb, cb, 2, PL.GREEDY), PL.plan(n, lb, cb, 0, PL.NONE),
           PL.plan(n, lb, cb, 0, PL.USER, [0, n - 2] if n > 2 else [0])]
    return out


@pytest.mark.parametrize("name", list(TINY))
def test_checkpointed_equals_full_storage(name):
    d = synth.make(TINY[name])
    chain = nets.Chain(d["structure"], d["params"])
    loss, grads = nets.full_storage_step(chain, d["input"], d["target"])
    n = chain.n
    for p in _plans(n):
        l2, g2, fwd = SCH.segment_step(chain, d["input"], d["target"], p)
        assert l2 == loss
        _same(grads, g2)
        assert fwd == PL.unit_forwards(p)
        if p.mode != PL.NONE and not p.keep_last:
            assert fwd == 2 * n
    l3, g3, fwd, live = SCH.recursive_step(chain, d["input"], d["target"])
    assert l3 == loss
    _same(grads, g3)
    p = PL.plan(n, [1] * n, [1] * (n - 1) + [0], 0, PL.RECURSIVE)
    assert fwd == n + p.extra_forwards
    assert live == math.ceil(math.log2(n))


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16, 32])
def test_recursive_counts_powers_of_two(n):
    cfg = dict(kind="mlp", depth=n, width=4, batch=2, seed=40 + n, w_var=0.1)
    d = synth.make(cfg)
    chain = nets.Chain(d["structure"], d["params"])
    _, _, fwd, live = SCH.recursive_step(chain, d["input"], d["target"])
    if n >= 2:
        assert fwd - n == n * (int(math.log2(n)) + 1) // 2
        assert live == int(math.log2(n))
    else:
        assert fwd == 2


def test_sqrt_plan_on_cfg_shapes_accounting():
    """The 64-block MLP at width 256, batch 64 with a checkpoint every 8 blocks:
    7 kept boundaries, a 8-block arena and 3 gradient buffers of 64 KiB."""
    st = synth.structure(synth.WORKLOADS["mlp64"])
    b, a, q = SZ.tables(st)
    lb, cb = SZ.layer_and_cut_bytes(st)
    p = PL.plan(st.n, lb, cb, 8, PL.SQRT)
    acc = PL.account(p, b, a, q)
    assert p.cuts == [7, 15, 23, 31, 39, 47, 55]
    assert (acc.ckpt, acc.arena, acc.grad) == (7 * 65536, 16 * 65536, 3 * 65536)
    none = PL.account(PL.plan(st.n, lb, cb, 0, PL.NONE), b, a, q)
    assert none.peak == 128 * 65536 + 3 * 65536


@pytest.mark.parametrize("k", [2, 3, 5])
def test_recursive_fanout_equals_full_storage(k):
    """Section 4.4 with k splits per level: same bits as full storage, the
    planner's unit-forward count, and k log_{k+1} n live boundaries at n = (k+1)^2."""
    n = (k + 1) ** 2
    cfg = dict(kind="mlp", depth=n, width=4, batch=2, seed=70 + k, w_var=0.1)
    d = synth.make(cfg)
    chain = nets.Chain(d["structure"], d["params"])
    loss, grads = nets.full_storage_step(chain, d["input"], d["target"])
    l3, g3, fwd, live = SCH.recursive_step(chain, d["input"], d["target"], k)
    assert l3 == loss
    _same(grads, g3)
    p = PL.plan(n, [1] * n, [1] * (n - 1) + [0], k, PL.RECURSIVE)
    assert fwd == n + p.extra_forwards
    assert live == 2 * k
    for name in ("lstm", "cnn", "bottleneck"):
        d = synth.make(TINY[name])
        chain = nets.Chain(d["structure"], d["params"])
        loss, grads = nets.full_storage_step(chain, d["input"], d["target"])
        l3, g3, fwd, _ = SCH.recursive_step(chain, d["input"], d["target"], k)
        assert l3 == loss
        _same(grads, g3)
        m = chain.n
        assert fwd == m + PL.plan(m, [1] * m, [1] * (m - 1) + [0], k, PL.RECURSIVE).extra_forwards
