"""Pins of the oracle's planners and accounting (CPU only).

* Alg. 3 hand-traced on a small size vector (tests/golden/greedy_small.json).
* Brute force over every cut set for n <= 14: the planner's x, y and PEAK are
  those of the cut set it returns, and for a uniform chain the best PEAK over
  all cut sets has the closed form min_k [(k-1) + 2 ceil(n/k) + 3] b, reached by
  the sqrt(n) plan at perfect squares (section 4.3, Eq. 1).
* Alg. 3 invariants: every cut is the first candidate where the running sum
  exceeds B; the number of cuts never grows with B; B = 0 cuts every candidate
  (of non-zero size); B >= total gives a single segment.
* Growth: the sqrt(n) plan's PEAK is (k - 1 + 2s + 3) b on a uniform chain, so
  PEAK/sqrt(n) stays bounded; the recursive plan keeps ceil(log2 n) boundaries
  (Eq. 3 with k = 1) and PEAK = (ceil(log2 n) + 6) b.
* Recompute: one-level plans run exactly 2n unit forwards (one extra forward
  pass, section 4.3); the recursive plan runs n + n(log2 n + 1)/2 for powers of
  two.
* Fan-out k (section 4.4, g(n) = k + g(n/(k+1))): for n = (k+1)^p on a uniform
  chain the recursion stores k p boundaries at most (k log_{k+1} n), PEAK is
  (k p + 6) b for p >= 2 and the extra unit forwards solve R(L) = L k/(k+1) + (k+1)
  R(L/(k+1)), R(1) = 1, i.e. n (1 + (p - 1) k/(k+1)).  With k >= n - 1 the
  top level stores every boundary: the accounting equals that of the
  one-level plan cutting at every unit (a separate code path), for any sizes.
* The per-unit byte tables agree with the nbytes of the tensors the float32
  oracle actually keeps.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import synth
from oracle import planner as PL
from oracle import sizes as SZ
from oracle import nets, units as U

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _uniform(n, b=256):
    return [b] * (n + 1), [b] * n, [b] * n


def _lc(b, a):
    n = len(a)
    return [a[i] + b[i + 1] for i in range(n)], [b[i + 1] for i in range(n - 1)] + [0]


def test_greedy_hand_traced_golden():
    with open(os.path.join(GOLDEN, "greedy_small.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        p = PL.plan(len(c["layer_bytes"]), c["layer_bytes"], c["cut_bytes"], c["B"], PL.GREEDY)
        assert p.cuts == c["cuts"] and p.x == c["x"] and p.y == c["y"], c


def _all_cut_sets(n):
    for r in range(n):
        for s in itertools.combinations(range(n - 1), r):
            yield list(s)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 8, 9, 12, 14])
def test_brute_force_random_sizes(n):
    rng = np.random.default_rng(n)
    b = [int(v) * 256 for v in rng.integers(1, 9, n + 1)]
    a = [int(v) * 256 for v in rng.integers(0, 9, n)]
    q = [int(v) * 256 for v in rng.integers(1, 9, n)]
    lb, cb = _lc(b, a)
    costs = {}
    for cuts in _all_cut_sets(n):
        p = PL.plan(n, lb, cb, 0, PL.USER, cuts)
        costs[tuple(cuts)] = (PL.account(p, b, a, q).peak, PL.xy_of_cuts(lb, cb, cuts))
    best = min(v[0] for v in costs.values())
    for mode, budget in [(PL.SQRT, 0), (PL.GREEDY, sum(lb) // 4), (PL.GREEDY, 0), (PL.NONE, 0)]:
        p = PL.plan(n, lb, cb, budget, mode)
        acc = PL.account(p, b, a, q)
        if mode != PL.NONE:
            peak, (x, y) = costs[tuple(p.cuts)]
            assert acc.peak == peak and (p.x, p.y) == (x, y)
        assert acc.peak >= best


@pytest.mark.parametrize("n", [2, 4, 7, 9, 13, 14])
def test_brute_force_uniform_closed_form(n):
    bsz = 256
    b, a, q = _uniform(n, bsz)
    lb, cb = _lc(b, a)
    best = min(PL.account(PL.plan(n, lb, cb, 0, PL.USER, c), b, a, q).peak for c in _all_cut_sets(n))
    closed = min((k - 1) + 2 * math.ceil(n / k) + 3 for k in range(1, n + 1)) * bsz
    assert best == closed
    if math.isqrt(n) ** 2 == n:
        p = PL.plan(n, lb, cb, 0, PL.SQRT)
        assert PL.account(p, b, a, q).peak == closed


def test_greedy_invariants():
    rng = np.random.default_rng(3)
    for trial in range(200):
        n = int(rng.integers(1, 40))
        lb = [int(v) for v in rng.integers(0, 1000, n)]
        cb = [int(v) if rng.random() < 0.7 else 0 for v in rng.integers(1, 500, n)]
        cb[-1] = 0
        prev = None
        for B in sorted(set([0, 1, 10, 100, 1000, 5000, sum(lb), sum(lb) + 1] +
                            [int(v) for v in rng.integers(0, sum(lb) + 2, 5)])):
            p = PL.plan(n, lb, cb, B, PL.GREEDY)
            # every cut is the first candidate past the budget since the last cut
            start = 0
            for c in p.cuts:
                run = 0
                for i in range(start, c + 1):
                    run += lb[i]
                    if i < c:
                        assert not (cb[i] > 0 and run > B)
                assert cb[c] > 0 and run > B
                start = c + 1
            run = 0
            for i in range(start, n):
                run += lb[i]
                assert not (cb[i] > 0 and run > B)
            if prev is not None:
                assert len(p.cuts) <= prev
            prev = len(p.cuts)
            if B >= sum(lb):
                assert p.cuts == []


def test_greedy_zero_budget_cuts_every_candidate():
    n = 10
    lb = [5] * n
    cb = [1] * (n - 1) + [0]
    assert PL.plan(n, lb, cb, 0, PL.GREEDY).cuts == list(range(n - 1))


@pytest.mark.parametrize("n", [16, 64, 256, 1024, 4096, 16384])
def test_sqrt_growth(n):
    bsz = 1024
    b, a, q = _uniform(n, bsz)
    lb, cb = _lc(b, a)
    p = PL.plan(n, lb, cb, 0, PL.SQRT)
    s = PL.ceil_isqrt(n)
    k = len(p.segments())
    assert k == math.ceil(n / s)
    acc = PL.account(p, b, a, q)
    assert acc.peak == (k - 1 + 2 * s + 3) * bsz
    assert acc.peak / (math.sqrt(n) * bsz) <= 4.0
    assert PL.unit_forwards(p) == 2 * n


@pytest.mark.parametrize("n", [1, 2, 3, 5, 6, 7, 16, 100, 1024, 16384])
def test_recursive_growth(n):
    bsz = 512
    b, a, q = _uniform(n, bsz)
    lb, cb = _lc(b, a)
    p = PL.plan(n, lb, cb, 0, PL.RECURSIVE)
    acc = PL.account(p, b, a, q)
    depth = math.ceil(math.log2(n)) if n > 1 else 0
    assert acc.ckpt == depth * bsz
    if n >= 3:
        assert acc.peak == (depth + 6) * bsz
    if n >= 2 and n & (n - 1) == 0:
        assert p.extra_forwards == n * (int(math.log2(n)) + 1) // 2
    if n == 1024:
        assert p.extra_forwards == 5632
    if n == 16384:
        assert p.extra_forwards == 122880


def test_keep_last_and_none():
    n = 12
    b, a, q = _uniform(n)
    lb, cb = _lc(b, a)
    p = PL.plan(n, lb, cb, 4, PL.SQRT, flags=PL.FLAG_KEEP_LAST)
    assert p.cuts == [3, 7] and p.extra_forwards == 8
    p0 = PL.plan(n, lb, cb, 0, PL.NONE)
    assert p0.extra_forwards == 0 and p0.cuts == []
    acc = PL.account(p0, b, a, q)
    assert acc.ckpt == 0 and acc.arena == sum(lb)


def test_errors():
    with pytest.raises(PL.PlanError):
        PL.plan(0, [], [], 0, PL.SQRT)
    with pytest.raises(PL.PlanError):
        PL.plan(3, [1, 1, 1], [1, 1, 1], 0, PL.SQRT)           # last unit marked as a cut
    with pytest.raises(PL.PlanError):
        PL.plan(4, [1] * 4, [1, 1, 1, 0], 0, PL.USER, [1, 0])  # unsorted
    with pytest.raises(PL.PlanError):
        PL.plan(4, [1] * 4, [1, 1, 1, 0], 0, PL.USER, [3])     # >= n-1
    with pytest.raises(PL.PlanError):
        PL.plan(4, [1] * 4, [1, 0, 1, 0], 0, PL.USER, [1])     # not a candidate
    with pytest.raises(PL.Unsupported):
        PL.plan(4, [1] * 4, [1, 0, 1, 0], 0, PL.RECURSIVE)
    with pytest.raises(PL.PlanError):
        PL.plan(4, [1] * 4, [1, 1, 1, 0], 0, 99)


def test_serialize_layout():
    p = PL.plan(5, [10] * 5, [4, 4, 4, 4, 0], 2, PL.SQRT)
    blob = p.serialize()
    assert blob[:4] == b"CKPL"
    assert len(blob) == 28 + 4 * len(p.cuts) + 24
    assert p.cuts == [1, 3]


@pytest.mark.parametrize("cfg", [dict(kind="mlp", depth=5, width=16, batch=4, seed=1),
                                 dict(kind="resnet_basic", blocks_per_stage=2, base=4, batch=2,
                                      image=8, classes=3, seed=2),
                                 dict(kind="resnet_basic", blocks_per_stage=2, base=4, batch=2,
                                      image=8, classes=3, seed=2, drop_bn_relu=1),
                                 dict(kind="resnet_bottleneck", stage_blocks=(2, 1), widths=(8, 16),
                                      expansion=4, stem_channels=8, image=16, batch=2, classes=5,
                                      seed=3),
                                 dict(kind="resnet_bottleneck", stage_blocks=(2, 1), widths=(8, 16),
                                      expansion=4, stem_channels=8, image=16, batch=2, classes=5,
                                      seed=3, drop_bn_relu=1),
                                 dict(kind="lstm", T=3, batch=4, input=8, hidden=16, vocab=24,
                                      seed=4)])
def test_size_tables_match_kept_tensors(cfg):
    """a_i and b_{i+1} equal the aligned bytes of what the oracle keeps, each
    tensor counted in the dtype the static layout stores it in: bf16 for the
    bottleneck net's activations and the LSTM's h, fp32 otherwise (batch-norm
    (mean, rstd) pairs, which the CNNs hold for the whole step, in the
    layout's fixed buffers instead of a_i).  The bottleneck stem's max-pool window
    choice ("arg") is not kept: the backward finds the window's first maximum
    again from the pooled output.  The drop bn-relu layouts keep no relu(bn(.))
    output of a block (the basic block's r1, the bottleneck's r1 and r2)."""
    d = synth.make(cfg)
    kind = cfg["kind"]
    chain = nets.Chain(d["structure"], d["params"], U.Prec(np.float32, kind == "resnet_bottleneck"))
    b, a, q = SZ.tables(d["structure"])
    drop = cfg.get("drop_bn_relu")

    def nbytes(name, v, half=False):
        return SZ.align((2 if half else 4) * v.size)

    def boundary(x):
        if kind == "lstm":                # (h bf16, c fp32)
            return nbytes("h", x[0], True) + nbytes("c", x[1])
        return nbytes("x", x, kind == "resnet_bottleneck")

    x = chain.x0(d["input"])
    assert boundary(x) == b[0]
    stats_kept = 0
    for i in range(chain.n):
        y, saved, _ = chain.units[i].fwd(x, chain.P(i), chain.ext(i, d["input"], d["target"]))
        kept = 0
        if kind == "lstm":                # the four gates as one [B, 4H] block, then dlog
            kept = SZ.align(sum(4 * saved[g].size for g in "ifgo")) + nbytes("dlog", saved["dlog"])
        else:
            for nm, v in saved.items():
                if nm == "arg" or (drop and nm in ("r1", "r2")):
                    continue
                if isinstance(v, tuple):  # BN (mean, rstd): held step-long, in the fixed buffers
                    stats_kept += SZ.align(sum(4 * t.size for t in v))
                    continue
                kept += nbytes(nm, v, kind == "resnet_bottleneck")
        assert kept == a[i], (i, kept, a[i])
        assert boundary(y) == b[i + 1]
        x = y
    # the batch-norm statistics of every unit are the layout's fixed buffers
    assert SZ.grad_layout(d["structure"])[1] == (stats_kept if kind.startswith("resnet") else
                                                 SZ.grad_layout(d["structure"])[1])


# ---- appendix-A search over the budget ----------------------------------

def test_search_hand_traced_golden():
    with open(os.path.join(GOLDEN, "search_small.json")) as f:
        g = json.load(f)
    lb, cb = g["layer_bytes"], g["cut_bytes"]
    _, x, y = PL.greedy_alg3(lb, cb, 0)
    assert (x, y) == (g["x0"], g["y0"])
    assert math.isqrt(x * y) == g["b0"]
    assert PL.search_candidates(lb, cb) == g["candidates"]
    for B, cuts in g["cuts"].items():
        assert PL.plan(len(lb), lb, cb, int(B), PL.GREEDY).cuts == cuts


@pytest.mark.parametrize("n,s,c", [(16, 1000, 300), (100, 4096, 512), (334, 77, 5)])
def test_search_candidates_closed_form_uniform(n, s, c):
    """Uniform layers: B = 0 keeps all n-1 candidates, x = (n-1) c, y = s."""
    lb, cb = [s] * n, [c] * (n - 1) + [0]
    b0 = math.isqrt((n - 1) * c * s)
    cands = PL.search_candidates(lb, cb)
    assert b0 in cands and len(cands) <= 7
    assert min(cands) == math.isqrt(b0 * b0 // 2) == math.floor(b0 / math.sqrt(2))
    assert max(cands) == math.isqrt(2 * b0 * b0)
    assert all(b0 / math.sqrt(2) - 1 <= B <= math.sqrt(2) * b0 for B in cands)


@pytest.mark.parametrize("seed", range(12))
def test_search_returns_lowest_exact_peak(seed):
    rng = np.random.default_rng(4000 + seed)
    n = int(rng.integers(1, 40))
    b = [int(v) for v in rng.integers(1, 5000, n + 1)]
    a = [int(v) for v in rng.integers(0, 9000, n)]
    q = [int(v) for v in rng.integers(0, 3000, n)]
    lb = [a[i] + b[i + 1] for i in range(n)]
    cb = [b[i + 1] if rng.random() < 0.8 else 0 for i in range(n - 1)] + [0]
    flags = PL.FLAG_KEEP_LAST if seed % 2 else 0
    p, B, peak = PL.search(n, lb, cb, b, a, q, None, 0, flags)
    peaks = {C: PL.account(PL.plan(n, lb, cb, C, PL.GREEDY, flags=flags), b, a, q).peak
             for C in PL.search_candidates(lb, cb)}
    assert peak == min(peaks.values())
    assert B == min(C for C, v in peaks.items() if v == peak)
    assert p.serialize() == PL.plan(n, lb, cb, B, PL.GREEDY, flags=flags).serialize()
    # never worse than the plain B0 run it refines
    b0 = math.isqrt(PL.greedy_alg3(lb, cb, 0)[1] * PL.greedy_alg3(lb, cb, 0)[2])
    assert peak <= peaks[b0]


@pytest.mark.parametrize("k", [1, 2, 3, 4, 7])
def test_recursive_fanout_closed_forms(k):
    bsz = 256
    for p in range(1, 8):
        n = (k + 1) ** p
        if n > 40000:
            break
        b, a, q = _uniform(n, bsz)
        lb, cb = _lc(b, a)
        pl = PL.plan(n, lb, cb, k, PL.RECURSIVE)
        assert pl.fanout == k
        acc = PL.account(pl, b, a, q)
        assert acc.ckpt == k * p * bsz, (k, p)
        if p >= 2:  # some sweep then holds a unit's input, internals and output
            assert acc.peak == (k * p + 6) * bsz, (k, p)
        # n (1 + (p - 1) k / (k + 1)), exact in integers
        assert pl.extra_forwards * (k + 1) == n * (k + 1 + (p - 1) * k), (k, p)


def test_recursive_fanout_one_is_the_default():
    n = 37
    b, a, q = _uniform(n)
    lb, cb = _lc(b, a)
    p0 = PL.plan(n, lb, cb, 0, PL.RECURSIVE)
    p1 = PL.plan(n, lb, cb, 1, PL.RECURSIVE)
    assert p0.serialize() == p1.serialize() and p0.fanout == 1


@pytest.mark.parametrize("n", [2, 3, 5, 9, 14])
def test_recursive_wide_fanout_is_every_cut(n):
    rng = np.random.default_rng(n)
    for _ in range(5):
        b = [int(v) for v in rng.integers(1, 1000, n + 1)]
        a = [int(v) for v in rng.integers(0, 1000, n)]
        q = [int(v) for v in rng.integers(0, 1000, n)]
        lb, cb = _lc(b, a)
        for k in (n - 1, n, 3 * n):
            pr = PL.plan(n, lb, cb, k, PL.RECURSIVE)
            assert PL.rec_splits(0, n, k) == list(range(1, n))
            pu = PL.plan(n, lb, cb, 0, PL.USER, list(range(n - 1)))
            ar, au = PL.account(pr, b, a, q), PL.account(pu, b, a, q)
            assert (ar.ckpt, ar.arena, ar.grad) == (au.ckpt, au.arena, au.grad)
            assert pr.extra_forwards == pu.extra_forwards == n


@pytest.mark.parametrize("k", [1, 2, 3, 5])
def test_rec_parts_cover_the_range(k):
    for lo in range(0, 4):
        for L in range(2, 40):
            parts = PL.rec_parts(lo, lo + L, k)
            assert parts[0][0] == lo and parts[-1][1] == lo + L
            assert all(p < q for (p, q) in parts)
            assert all(parts[t][1] == parts[t + 1][0] for t in range(len(parts) - 1))
            assert len(parts) == min(k + 1, L)
            sizes = [q - p for (p, q) in parts]
            assert max(sizes) - min(sizes) <= 1
