"""Pins of the oracle's gradient-graph construction (Alg. 2) and static
allocator (section 3), CPU only.

* Section 3's two-layer network traced by hand for every strategy and for a
  mirrored plan (tests/golden/graph_small.json): execution order, tags, peak.
* Random DAGs, every strategy, mirror counts 0..2:
  - every node runs after its inputs; without mirrors the order is the
    forward graph followed by one gradient node per forward node, last to
    first;
  - no two outputs that are live at the same time share a memory block, except
    an in-place write taking over its own first input at the moment that
    input dies; NONE never shares, INPLACE shares only in place;
  - the peak is at least the largest total of simultaneously live outputs and
    NONE's peak is the sum of all outputs;
  - value check: with each operator a distinct hash of its inputs' values,
    every mirror node reproduces its forward node's value, and every gradient
    node reads nodes whose values are those of v's output / inputs and the
    gradient nodes of v's successors;
  - v gets exactly m(v) mirror nodes, chained through the rounds.
* Segmented mirror plans on a chain schedule every mirror (each is needed).
"""
import json
import os

import numpy as np
import pytest

from oracle import graph as G
from synth import graphs as SG

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FLAG = {"-": 0, "GRAD_IN": G.GRAD_IN, "INPLACE|GRAD_OUT": G.INPLACE | G.GRAD_OUT,
        "GRAD_OUT": G.GRAD_OUT}
STRAT = {"NONE": G.ALLOC_NONE, "INPLACE": G.ALLOC_INPLACE, "SHARE": G.ALLOC_SHARE}


def test_two_layer_hand_traced():
    with open(os.path.join(GOLDEN, "graph_small.json")) as f:
        gold = json.load(f)
    flags = [FLAG[x] for x in gold["flags"]]
    for c in gold["cases"]:
        p = G.plan(gold["pred"], gold["out_bytes"], flags, c["mirror"], STRAT[c["strategy"]])
        assert p.order == c["order"], c["strategy"]
        assert p.peak == c["peak"], c["strategy"]
        if "tags" in c:
            assert {str(k): v for k, v in p.tag_of.items()} == c["tags"], c["strategy"]
        if "n_mirror" in c:
            assert p.n_mirror == c["n_mirror"]


def random_dag(rng, n, max_in=3, p_edge=0.5):
    pred = [[]]
    for v in range(1, n):
        k = int(rng.integers(1, max_in + 1)) if rng.random() < 0.9 else 0
        cands = list(range(v))
        # favour recent nodes, sometimes reach far back (skip connections)
        ins = sorted(set(int(max(0, v - 1 - rng.geometric(p_edge) + 1)) for _ in range(k)))
        ins = [u for u in ins if u in cands]
        if rng.random() < 0.2 and v > 2:
            ins.append(int(rng.integers(0, v)))
        pred.append(ins)
    out_bytes = [int(b) for b in rng.choice([0, 16, 32, 64, 128, 256], size=n, p=[.05, .2, .2, .25, .2, .1])]
    flags = [int(f) for f in rng.integers(0, 8, size=n)]
    mirror = [int(m) for m in rng.choice([0, 1, 2], size=n, p=[.5, .35, .15])]
    return pred, out_bytes, flags, mirror


def _intervals(p):
    pos = {w: i for i, w in enumerate(p.order)}
    last = {w: pos[w] for w in p.order}
    for w in p.order:
        for i in p.nodes[w].inputs:
            last[i] = max(last[i], pos[w])
    return pos, last


def _check_valid(p, strategy):
    pos, last = _intervals(p)
    for w in p.order:
        for i in p.nodes[w].inputs:
            assert pos[i] < pos[w]
    by_tag = {}
    for w in p.order:
        t = p.tag_of[w]
        if p.nodes[w].bytes == 0:
            assert t == -1
            continue
        assert t >= 0 and p.tag_bytes[t] >= p.nodes[w].bytes
        by_tag.setdefault(t, []).append(w)
    for t, ws in by_tag.items():
        ws.sort(key=lambda w: pos[w])
        if strategy == G.ALLOC_NONE:
            assert len(ws) == 1
        for a, b in zip(ws, ws[1:]):
            in_place = p.nodes[b].inplace and p.nodes[b].inputs and p.nodes[b].inputs[0] == a
            if in_place:
                assert last[a] == pos[b]          # the input dies at the in-place write
            else:
                assert strategy == G.ALLOC_SHARE
                assert last[a] < pos[b]           # strictly dead before reuse


@pytest.mark.parametrize("seed", range(12))
def test_random_dags_valid_allocation(seed):
    rng = np.random.default_rng(seed)
    pred, ob, fl, mi = random_dag(rng, int(rng.integers(3, 40)))
    base = None
    for strategy in (G.ALLOC_NONE, G.ALLOC_INPLACE, G.ALLOC_SHARE):
        p = G.plan(pred, ob, fl, mi, strategy)
        _check_valid(p, strategy)
        if strategy == G.ALLOC_NONE:
            assert p.peak == sum(p.nodes[w].bytes for w in p.order)
            base = p.order
        else:
            assert p.order == base                # the order does not depend on the allocator


def test_live_bytes_lower_bound():
    """Outputs live at the same step occupy distinct blocks (an in-place
    writer and its input count once), so the sum of the blocks is at least the
    live total at every step."""
    rng = np.random.default_rng(99)
    for _ in range(30):
        pred, ob, fl, mi = random_dag(rng, int(rng.integers(3, 30)))
        p = G.plan(pred, ob, fl, mi, G.ALLOC_SHARE)
        pos, last = _intervals(p)
        for i, w in enumerate(p.order):
            live_tags = {p.tag_of[x] for x in p.order[:i + 1] if last[x] >= i and p.tag_of[x] >= 0}
            assert p.peak >= sum(p.tag_bytes[t] for t in live_tags)
            live = [x for x in p.order[:i + 1] if last[x] >= i and p.nodes[x].bytes > 0
                    and not (last[x] == i and p.tag_of.get(w) == p.tag_of[x] and x != w)]
            assert p.peak >= sum(p.nodes[x].bytes for x in live)


@pytest.mark.parametrize("seed", range(10))
def test_mirrors_recompute_the_same_values(seed):
    rng = np.random.default_rng(100 + seed)
    pred, ob, fl, mi = random_dag(rng, int(rng.integers(4, 30)))
    p = G.build(pred, ob, fl, mi)
    n = len(pred)
    salt = [int(x) for x in rng.integers(1, 1 << 30, size=n)]
    val = {}

    def f(v, ins):
        h = salt[v]
        for x in ins:
            h = (h * 1000003 + x) % (1 << 61)
        return h

    for w, nd in enumerate(p.nodes):
        if nd.kind in (G.FWD, G.MIRROR):
            val[w] = f(nd.of, [val[i] for i in nd.inputs])
    for w, nd in enumerate(p.nodes):
        if nd.kind == G.MIRROR:
            assert val[w] == val[nd.of]
    count = [0] * n
    for nd in p.nodes:
        if nd.kind == G.MIRROR:
            count[nd.of] += 1
    for v in range(n):
        assert count[v] == (mi[v] if pred[v] else 0)
    succ = [[] for _ in range(n)]
    for v in range(n):
        for u in pred[v]:
            if v not in succ[u]:
                succ[u].append(v)
    gnode = {nd.of: w for w, nd in enumerate(p.nodes) if nd.kind == G.GRAD}
    for v in range(n):
        nd = p.nodes[gnode[v]]
        k = len(succ[v])
        assert [p.nodes[i].of for i in nd.inputs[:k]] == succ[v]
        assert all(p.nodes[i].kind == G.GRAD for i in nd.inputs[:k])
        rest = nd.inputs[k:]
        want = ([val[v]] if fl[v] & G.GRAD_OUT else []) + \
               ([val[u] for u in pred[v]] if fl[v] & G.GRAD_IN else [])
        assert [val[i] for i in rest] == want
        assert nd.bytes == sum(ob[u] for u in pred[v])


def test_no_mirror_order_is_forward_then_reverse():
    g = SG.resnet_basic(2, 4, 2, 8, 3)
    p = G.build(g["pred"], g["bytes"], g["flags"], None)
    n = len(g["op"])
    assert p.order[:n] == list(range(n))
    assert [p.nodes[w].of for w in p.order[n:]] == list(range(n - 1, -1, -1))
    assert all(p.nodes[w].kind == G.GRAD for w in p.order[n:])


def test_segment_mirrors_are_all_scheduled():
    g = SG.mlp(16, 8, 2)
    m = SG.mirror_segments(g, 4)
    p = G.plan(g["pred"], g["bytes"], g["flags"], m, G.ALLOC_SHARE)
    assert p.n_mirror == sum(m)
    # a kept block output is never recomputed
    kept = set(g["block_out"][3::4])
    assert not any(p.nodes[w].kind == G.MIRROR and p.nodes[w].of in kept for w in p.order)


def test_errors():
    with pytest.raises(G.GraphError):
        G.build([[], [1]], [1, 1], [0, 0])          # not topological
    with pytest.raises(G.GraphError):
        G.build([[], [0]], [1, 1], [0, 0], [0, -1])
    with pytest.raises(G.GraphError):
        G.allocate(G.build([[]], [1], [0]), 7)
