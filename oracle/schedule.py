"""CPU executors of the checkpointed step, with a unit-forward counter.

TEST INFRASTRUCTURE ONLY (see the package header).

* ``segment_step`` follows Alg. 1: the forward pass keeps only each segment's
  input (temp[k]); the head gives g; then for every segment in reverse order
  the segment is re-run from its stored input into a local table (localtemp)
  and back-propagated unit by unit.  With keep_last the last segment's
  activations from the first forward are used instead of a re-run.
* ``recursive_step`` follows section 4.4 with k = 1: the first forward keeps
  the midpoint boundary; a range [a, b) of length > 1 is handled by running
  its first half forward from x_a, keeping x_m (m = a + floor((b-a)/2)),
  treating [m, b) the same way, dropping x_m and then treating [a, m); a single
  unit is re-run once and back-propagated.

Both return exactly the gradients of ``nets.full_storage_step`` (the paper
states that the optimisations give the same weight gradient, section 5.1),
since they call the same unit functions on the same values.

Parity: pinned by bit-identity against the full-storage step and by the
unit-forward counts 2n (one extra forward pass, section 4.3) and
n + n(log2 n + 1)/2 for powers of two (tests/test_oracle_schedule.py).
"""
from __future__ import annotations

from . import planner as PL
from .nets import Chain


class _Counter:
    def __init__(self):
        self.fwd = 0
        self.live_ckpts = 0
        self.max_live_ckpts = 0


def _fwd(chain: Chain, i, x, inp, target, cnt):
    cnt.fwd += 1
    return chain.units[i].fwd(x, chain.P(i), chain.ext(i, inp, target))


def _bwd_unit(chain, i, g, x, y, saved, inp, target, grads):
    g, ug = chain.units[i].bwd(g, x, y, saved, chain.P(i), chain.ext(i, inp, target),
                               need_dx=(i > 0))
    chain.add_unit_grads(grads, i, ug)
    return g


def segment_step(chain: Chain, inp, target, plan: PL.Plan):
    inp = chain.prec.cast(inp)
    cnt = _Counter()
    segs = plan.segments()
    temp = {}
    v = chain.x0(inp)
    loss = 0.0
    last_local = None
    for k, (lo, hi) in enumerate(segs):
        temp[k] = v
        keep = plan.keep_last and k == len(segs) - 1
        local = []
        for i in range(lo, hi):
            y, s, lp = _fwd(chain, i, v, inp, target, cnt)
            loss += lp
            if keep:
                local.append((v, y, s))
            v = y
        if keep:
            last_local = local
    hl, g, hgrads = chain.head(v, target)
    loss += hl
    grads = chain.zero_grads()
    for name, val in hgrads.items():
        grads[name] += val
    for k in range(len(segs) - 1, -1, -1):
        lo, hi = segs[k]
        if plan.keep_last and k == len(segs) - 1:
            local = last_local
        else:
            v = temp[k]
            local = []
            for i in range(lo, hi):
                y, s, _ = _fwd(chain, i, v, inp, target, cnt)
                local.append((v, y, s))
                v = y
        for i in range(hi - 1, lo - 1, -1):
            x, y, s = local[i - lo]
            g = _bwd_unit(chain, i, g, x, y, s, inp, target, grads)
    return loss, grads, cnt.fwd


def recursive_step(chain: Chain, inp, target, k: int = 1):
    """Section 4.4's recursion with k stored splits per level (parts from
    planner.rec_parts): forward a range up to its last split point storing the
    split boundaries, handle the parts last to first, drop each boundary once
    its part is done; a single unit is re-forwarded and back-propagated.
    Returns (loss, grads, unit forwards, the most boundaries stored at once)."""
    inp = chain.prec.cast(inp)
    cnt = _Counter()
    n = chain.n
    loss = 0.0
    grads = chain.zero_grads()
    state = {"g": None}

    def run_forward(lo, hi, x, keep, first=False):
        """Forward [lo, hi) from x; return (x_hi, {m: x_m for m in keep})."""
        nonlocal loss
        kept = {}
        v = x
        for i in range(lo, hi):
            v, _, lp = _fwd(chain, i, v, inp, target, cnt)
            if first:
                loss += lp  # the loss parts are taken from the first forward only
            if i + 1 in keep:
                kept[i + 1] = v
        return v, kept

    def handle(parts, x_lo, kept):
        for t in range(len(parts) - 1, -1, -1):
            p, q = parts[t]
            R(p, q, kept[p] if t > 0 else x_lo)
            if t > 0:
                del kept[p]
                cnt.live_ckpts -= 1

    def R(lo, hi, x_lo):
        if hi - lo == 1:
            y, s, _ = _fwd(chain, lo, x_lo, inp, target, cnt)
            state["g"] = _bwd_unit(chain, lo, state["g"], x_lo, y, s, inp, target, grads)
            return
        parts = PL.rec_parts(lo, hi, k)
        splits = [p for (p, _) in parts[1:]]
        _, kept = run_forward(lo, splits[-1], x_lo, set(splits))
        cnt.live_ckpts += len(splits)
        cnt.max_live_ckpts = max(cnt.max_live_ckpts, cnt.live_ckpts)
        handle(parts, x_lo, kept)

    x0 = chain.x0(inp)
    parts = PL.rec_parts(0, n, k) if n > 1 else [(0, 1)]
    splits = [p for (p, _) in parts[1:]]
    v, kept = run_forward(0, n, x0, set(splits), first=True)
    cnt.live_ckpts = len(splits)
    cnt.max_live_ckpts = cnt.live_ckpts
    hl, g, hgrads = chain.head(v, target)
    loss += hl
    for name, val in hgrads.items():
        grads[name] += val
    state["g"] = g
    if n == 1:
        R(0, 1, x0)
    else:
        handle(parts, x0, kept)
    return loss, grads, cnt.fwd, cnt.max_live_ckpts
