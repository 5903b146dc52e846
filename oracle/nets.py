"""Chain networks and the plain full-storage training step.

TEST INFRASTRUCTURE ONLY (see the package header).

A network is a chain of n units u_0..u_{n-1}; unit i maps x_i to x_{i+1}
(section 4.1 treats exactly this linear chain).  The head turns x_n into the
loss and its gradient g (the ``gradient(v, label)`` step of Alg. 1).  The
full-storage step keeps every unit's saved tensors from one forward pass and
then runs the backward pathway in reverse topological order (section 3), i.e.
unit n-1 down to unit 0.  Gradients of shared parameters (the LSTM's) are
summed in that same backward order.

Parity: pinned by finite differences of the whole step on tiny networks
(tests/test_oracle_units.py).
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

from . import units as U


class Chain:
    """Units + head of one workload, bound to a parameter mapping."""

    def __init__(self, structure, params: Dict[str, np.ndarray], prec: U.Prec = U.F64):
        self.st = structure
        self.prec = prec
        self.params = {k: prec.cast(v) for k, v in params.items()}
        self.kind = structure.kind
        self.units: List = []
        self.local: List[Dict[str, str]] = []      # unit-local name -> global name
        cfg = structure.cfg
        if self.kind == "lstm":
            scale = 1.0 / (cfg["T"] * cfg["batch"])
            shared = {k: k for k in ("W_x", "W_h", "b", "W_o", "b_o")}
            for _ in structure.units:
                self.units.append(U.LSTMStep(cfg["hidden"], scale, prec))
                self.local.append(shared)
        else:
            for i, u in enumerate(structure.units):
                names = {nm.split(".", 1)[1]: nm for nm, _, _ in u.params}
                self.local.append(names)
                if u.kind == "mlp":
                    self.units.append(U.MLPBlock(prec))
                elif u.kind == "stem3":
                    self.units.append(U.Stem3(prec))
                elif u.kind == "basic":
                    self.units.append(U.BasicBlock(u.stride, u.cin, u.cout, prec))
                elif u.kind == "stem7":
                    self.units.append(U.Stem7(prec))
                elif u.kind == "bottleneck":
                    self.units.append(U.Bottleneck(u.stride, u.cin, u.width, u.cout, u.proj, prec))
                else:
                    raise ValueError(u.kind)

    @property
    def n(self) -> int:
        return len(self.units)

    def P(self, i):
        return {k: self.params[g] for k, g in self.local[i].items()}

    # ---- per-unit external inputs ------------------------------------
    def ext(self, i, inp, target):
        if self.kind == "lstm":
            return (inp[i], target[i])
        return None

    def x0(self, inp):
        if self.kind == "lstm":
            B, H = inp.shape[1], self.st.cfg["hidden"]
            z = np.zeros((B, H), dtype=self.prec.dtype)
            return (z, z.copy())
        return self.prec.st(self.prec.cast(inp))

    # ---- head ---------------------------------------------------------
    def head(self, xn, target):
        """loss, g (gradient w.r.t. x_n), head parameter grads."""
        if self.kind == "mlp":
            loss, g = U.mse_head(xn, self.prec.cast(target))
            return loss, g, {}
        if self.kind == "lstm":
            h, c = xn
            return 0.0, (np.zeros_like(h), np.zeros_like(c)), {}
        loss, g, grads = U.pool_fc_ce_head(xn, self.params["head.W"], self.params["head.b"],
                                           target, self.prec)
        return loss, g, {"head.W": grads["W"], "head.b": grads["b"]}

    # ---- gradient bookkeeping -----------------------------------------
    def zero_grads(self):
        return {k: np.zeros_like(v) for k, v in self.params.items()}

    def add_unit_grads(self, total, i, grads):
        for k, v in grads.items():
            total[self.local[i][k]] += v


def full_storage_step(chain: Chain, inp, target):
    """Forward storing every unit's saved tensors, head, backward n-1..0.

    Returns (loss, grads) with grads keyed by global parameter name.
    """
    inp = chain.prec.cast(inp) if chain.kind != "lstm" else chain.prec.cast(inp)
    xs = [chain.x0(inp)]
    saved = []
    loss = 0.0
    for i in range(chain.n):
        y, s, lp = chain.units[i].fwd(xs[i], chain.P(i), chain.ext(i, inp, target))
        xs.append(y)
        saved.append(s)
        loss += lp
    hl, g, hgrads = chain.head(xs[-1], target)
    loss += hl
    grads = chain.zero_grads()
    for k, v in hgrads.items():
        grads[k] += v
    for i in range(chain.n - 1, -1, -1):
        g, ug = chain.units[i].bwd(g, xs[i], xs[i + 1], saved[i], chain.P(i),
                                   chain.ext(i, inp, target), need_dx=(i > 0))
        chain.add_unit_grads(grads, i, ug)
    return loss, grads
