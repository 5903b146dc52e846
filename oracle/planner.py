"""Checkpoint planners and the memory accounting of a static plan.

TEST INFRASTRUCTURE ONLY (see the package header).

Notation.  The chain has n units; unit i maps x_i to x_{i+1}.  For each unit
the caller gives ``layer_bytes[i]`` -- the bytes the unit holds while its
segment is re-run (its saved internals plus its output; Alg. 3's
"size-of-output" at unit granularity) -- and ``cut_bytes[i]`` -- the bytes of
x_{i+1}, kept when the chain is cut after unit i, or 0 when x_{i+1} is not a
candidate split point (Alg. 3's set C).  The last unit is never a candidate:
its output feeds the loss directly (Alg. 1).

A cut c means: store x_{c+1} (Alg. 3 sets m(v) = 0 on that node) and start a
new segment at unit c+1.  Segments are half-open [begin, end) as in Alg. 1.

Modes:
* NONE      -- one segment, forward activations kept (no recomputation).
* SQRT      -- section 4.3, Eq. 1: k = ceil(sqrt(n)) equal segments (stride s,
               cuts at s-1, 2s-1, ... below n-1); an explicit stride may be
               given in ``budget``.  A target that is not a candidate moves to
               the next candidate.
* GREEDY    -- Alg. 3: walk the units in order accumulating temp; at a
               candidate where temp > B, cut, add the cut's bytes to x, raise y
               to temp and reset temp to 0.  x and y are returned exactly as
               Alg. 3 computes them (y only sees segments that end at a cut).
* RECURSIVE -- section 4.4 (Eq. 2-3) with k stored splits per level (``budget``
               gives k; 0 means k = 1): a range [lo, lo + L) with L > 1 is
               split into at most k + 1 parts at lo + floor(j L / (k+1)),
               j = 1..k (repeated or end points dropped); one forward sweep
               stores the split boundaries, then the parts are handled the
               same way from last to first, each split point dropped once its
               part is done; a single unit is re-forwarded once.  The stored
               boundaries follow g(n) = k + g(n / (k+1)), i.e. k log_{k+1} n.
* USER      -- an explicit cut list (the user-set mirror attribute of
               section 4.5).

Flag KEEP_LAST: the last segment keeps the activations of the first forward
instead of recomputing them (the literal Alg. 1 re-runs every segment, so
without the flag a one-level plan costs exactly n extra unit forwards).  NONE
always keeps them.

Accounting (exact bytes of the executor's static layout; the paper reports the
exact feature-map cost of a static plan, excluding parameters and temporary
operator workspace, section 5.1):
* CKPT  -- stored boundaries.  One-level: sum of b_{c+1} over cuts.
           Recursive: the largest total of simultaneously stored split points.
* ARENA -- the largest of (a) every forward-sweep unit's transient need
           (input if it lives in the arena) + internals + (output if it is not
           stored), and (b) every re-run segment's sum of internals + outputs.
* GRAD  -- two gradient slots (each the size of the largest boundary's
           gradient: max_{1<=i<=n} b_i unless the unit kind says otherwise),
           one scratch of max q_i, plus any fixed gradient buffers of the
           unit kind (the LSTM's weight-gradient chunk buffers).
* PEAK  -- CKPT + ARENA + GRAD.

Parity: pinned by brute force over all cut sets for n <= 16, Alg. 3
invariants, and the closed forms of Eq. 1 and Eq. 3 (tests/test_oracle_planner.py).
"""
from __future__ import annotations

import math
import struct
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

NONE, SQRT, GREEDY, RECURSIVE, USER = 0, 1, 2, 3, 4
FLAG_KEEP_LAST = 1
MAGIC = b"CKPL"
VERSION = 2


class PlanError(ValueError):
    pass


class Unsupported(PlanError):
    pass


@dataclass
class Plan:
    mode: int
    n: int
    cuts: List[int] = field(default_factory=list)
    x: int = 0
    y: int = 0
    extra_forwards: int = 0
    keep_last: bool = False
    fanout: int = 0          # RECURSIVE: k stored splits per level; 0 otherwise

    def segments(self):
        """Half-open [begin, end) segments of a one-level plan."""
        out, b = [], 0
        for c in self.cuts:
            out.append((b, c + 1))
            b = c + 1
        out.append((b, self.n))
        return out

    def serialize(self) -> bytes:
        body = struct.pack("<4sIIIIII", MAGIC, VERSION, self.mode, 1 if self.keep_last else 0,
                           self.fanout, self.n, len(self.cuts))
        body += struct.pack(f"<{len(self.cuts)}i", *self.cuts)
        body += struct.pack("<QQQ", self.x, self.y, self.extra_forwards)
        return body


def ceil_isqrt(n: int) -> int:
    r = math.isqrt(n)
    return r if r * r == n else r + 1


def xy_of_cuts(layer_bytes: Sequence[int], cut_bytes: Sequence[int], cuts: Sequence[int]):
    """Alg. 3's outputs for a given cut set: x = kept bytes, y = the largest
    segment total among segments that end at a cut."""
    x = sum(cut_bytes[c] for c in cuts)
    y, b = 0, 0
    for c in cuts:
        y = max(y, sum(layer_bytes[b:c + 1]))
        b = c + 1
    return x, y


def greedy_alg3(layer_bytes, cut_bytes, B):
    """Alg. 3, step by step."""
    temp = x = y = 0
    cuts = []
    for i in range(len(layer_bytes)):
        temp += layer_bytes[i]
        if cut_bytes[i] > 0 and temp > B:
            x += cut_bytes[i]
            y = max(y, temp)
            cuts.append(i)
            temp = 0
    return cuts, x, y


def sqrt_cuts(n, cut_bytes, stride):
    cuts = []
    j = 1
    while True:
        t = j * stride - 1
        if t >= n - 1:
            break
        c = t
        while c < n - 1 and cut_bytes[c] == 0:
            c += 1
        if c < n - 1 and (not cuts or c > cuts[-1]):
            cuts.append(c)
        j += 1
    return cuts


def rec_splits(lo: int, hi: int, k: int) -> List[int]:
    """The split points of [lo, hi) for fan-out k: lo + floor(j L / (k+1)) for
    j = 1..k, keeping those strictly inside the range, without repeats."""
    L = hi - lo
    pts = []
    for j in range(1, k + 1):
        m = lo + (j * L) // (k + 1)
        if lo < m < hi and (not pts or m > pts[-1]):
            pts.append(m)
    return pts


def rec_parts(lo: int, hi: int, k: int):
    """The parts [lo, m_1), [m_1, m_2), ..., [m_last, hi) of a split range."""
    e = [lo] + rec_splits(lo, hi, k) + [hi]
    return [(e[t], e[t + 1]) for t in range(len(e) - 1)]


def recursive_extra(n: int, k: int = 1) -> int:
    """Unit forwards done after the first full forward, by the recursion: a
    range of one unit is re-forwarded once; a longer range re-runs the sweep
    up to its last split point, then its parts."""
    def R(a, b):
        if b - a == 1:
            return 1
        parts = rec_parts(a, b, k)
        return (parts[-1][0] - a) + sum(R(p, q) for (p, q) in parts)
    if n == 1:
        return R(0, 1)
    return sum(R(p, q) for (p, q) in rec_parts(0, n, k))


def plan(n: int, layer_bytes: Sequence[int], cut_bytes: Sequence[int], budget: int, mode: int,
         user_cuts: Optional[Sequence[int]] = None, flags: int = 0) -> Plan:
    if n <= 0 or len(layer_bytes) != n or len(cut_bytes) != n:
        raise PlanError("n must be positive and both size arrays must have n entries")
    if any(v < 0 for v in layer_bytes) or any(v < 0 for v in cut_bytes):
        raise PlanError("sizes are unsigned")
    if cut_bytes[n - 1] != 0:
        raise PlanError("the last unit cannot be a cut")
    keep_last = bool(flags & FLAG_KEEP_LAST)
    if mode == NONE:
        return Plan(NONE, n, [], 0, 0, 0, True)
    if mode == SQRT:
        stride = budget if budget > 0 else ceil_isqrt(n)
        cuts = sqrt_cuts(n, cut_bytes, stride)
    elif mode == GREEDY:
        cuts, x, y = greedy_alg3(layer_bytes, cut_bytes, budget)
    elif mode == USER:
        cuts = list(user_cuts or [])
        for k, c in enumerate(cuts):
            if c < 0 or c >= n - 1 or cut_bytes[c] == 0 or (k and c <= cuts[k - 1]):
                raise PlanError("user cuts must be ascending candidates below n-1")
    elif mode == RECURSIVE:
        if any(cut_bytes[i] == 0 for i in range(n - 1)):
            raise Unsupported("the recursive schedule needs every boundary to be a candidate")
        k = budget if budget > 0 else 1
        if k >= 1 << 31:
            raise PlanError("the recursion fan-out must fit in 31 bits")
        return Plan(RECURSIVE, n, [], 0, 0, recursive_extra(n, k), False, k)
    else:
        raise PlanError(f"unknown mode {mode}")
    x, y = xy_of_cuts(layer_bytes, cut_bytes, cuts)
    p = Plan(mode, n, cuts, x, y, 0, keep_last)
    if keep_last:
        p.extra_forwards = cuts[-1] + 1 if cuts else 0
    else:
        p.extra_forwards = n
    return p


# --------------------------------------------------------------------------
# accounting
# --------------------------------------------------------------------------

@dataclass
class Accounting:
    ckpt: int
    arena: int
    grad: int

    @property
    def peak(self) -> int:
        return self.ckpt + self.arena + self.grad


def _sweep_needs(b, a, lo, hi, stored):
    """Transient arena need of each unit of a forward sweep over [lo, hi) whose
    first input is external; ``stored`` is the set of units whose output is kept
    outside the arena."""
    needs = []
    for i in range(lo, hi):
        in_arena = i > lo and (i - 1) not in stored
        out_arena = i not in stored
        needs.append((b[i] if in_arena else 0) + a[i] + (b[i + 1] if out_arena else 0))
    return needs


def grad_bytes(b, q, slot=None, extra=0):
    n = len(q)
    if slot is None:
        slot = max(b[1:n + 1])
    return 2 * slot + max(q) + extra


def account(p: Plan, b: Sequence[int], a: Sequence[int], q: Sequence[int], slot=None,
            extra: int = 0) -> Accounting:
    """b has n+1 entries (x_0..x_n), a and q have n entries; slot and extra
    describe the gradient buffers when they differ from the boundaries."""
    n = p.n
    assert len(b) == n + 1 and len(a) == n and len(q) == n
    G = grad_bytes(b, q, slot, extra)
    if p.mode == RECURSIVE:
        k = p.fanout
        arena = 0
        stack: List[int] = []
        ckpt_max = 0

        def handle_parts(parts):
            # split boundaries of parts[1:] are on the stack; the last part
            # is handled first and its boundary dropped after it
            nonlocal ckpt_max
            for t in range(len(parts) - 1, -1, -1):
                R(*parts[t])
                if t > 0:
                    stack.pop()

        def R(lo, hi):
            nonlocal arena, ckpt_max
            if hi - lo == 1:
                arena = max(arena, a[lo] + b[lo + 1])
                return
            parts = rec_parts(lo, hi, k)
            splits = [q for (q, _) in parts[1:]]
            arena = max(arena, *_sweep_needs(b, a, lo, splits[-1], {m - 1 for m in splits}))
            for m in splits:
                stack.append(b[m])
            ckpt_max = max(ckpt_max, sum(stack))
            handle_parts(parts)

        if n == 1:
            arena = max(arena, *_sweep_needs(b, a, 0, 1, set()))
            R(0, 1)
        else:
            parts = rec_parts(0, n, k)
            splits = [q for (q, _) in parts[1:]]
            arena = max(arena, *_sweep_needs(b, a, 0, n, {m - 1 for m in splits}))
            for m in splits:
                stack.append(b[m])
            ckpt_max = max(ckpt_max, sum(stack))
            handle_parts(parts)
        return Accounting(ckpt_max, arena, G)
    cuts = set(p.cuts)
    segs = p.segments()
    fwd_hi = segs[-1][0] if p.keep_last else n
    arena = 0
    if fwd_hi > 0:
        arena = max(_sweep_needs(b, a, 0, fwd_hi, cuts))
    for (lo, hi) in segs:
        arena = max(arena, sum(a[i] + b[i + 1] for i in range(lo, hi)))
    ckpt = sum(b[c + 1] for c in p.cuts)
    return Accounting(ckpt, arena, G)


def unit_forwards(p: Plan) -> int:
    return p.n + p.extra_forwards


# --------------------------------------------------------------------------
# search over Alg. 3's budget (appendix A)
# --------------------------------------------------------------------------

def search_candidates(layer_bytes: Sequence[int], cut_bytes: Sequence[int]) -> List[int]:
    """The budgets the appendix-A search tries: run Alg. 3 with B = 0 to get
    x (kept bytes) and y (largest segment), take B0 = floor(sqrt(x y)), then a
    six-point grid on [B0/sqrt(2), sqrt(2) B0].  Reading: the grid is evenly
    spaced between floor(B0/sqrt 2) and floor(sqrt(2) B0) (integer square
    roots, integer steps j (hi - lo) // 5), and B0 itself is a candidate too.
    Returned ascending, without repeats."""
    _, x, y = greedy_alg3(layer_bytes, cut_bytes, 0)
    b0 = math.isqrt(x * y)
    lo = math.isqrt(b0 * b0 // 2)
    hi = math.isqrt(2 * b0 * b0)
    grid = [lo + (hi - lo) * j // 5 for j in range(6)]
    return sorted(set(grid + [b0]))


def search(n: int, layer_bytes: Sequence[int], cut_bytes: Sequence[int], b: Sequence[int],
           a: Sequence[int], q: Sequence[int], slot=None, extra: int = 0, flags: int = 0):
    """Appendix A: the GREEDY plan of the candidate budget with the lowest
    exact PEAK of the static layout (ties: the smaller budget).  Returns
    (plan, budget, peak)."""
    best = None
    for B in search_candidates(layer_bytes, cut_bytes):
        p = plan(n, layer_bytes, cut_bytes, B, GREEDY, flags=flags)
        pk = account(p, b, a, q, slot, extra).peak
        if best is None or pk < best[2]:
            best = (p, B, pk)
    return best

