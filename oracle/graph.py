"""Gradient-graph construction with mirror nodes, and the static memory allocator.

TEST INFRASTRUCTURE ONLY (see the package header).

Forward graph.  Nodes 0..n-1 are listed in a topological order; ``pred[v]`` are
the nodes whose outputs v reads, ``out_bytes[v]`` the bytes of v's output,
``flags[v]`` says whether v's operator may write its output over its first
input (INPLACE) and what v's backward reads besides the incoming gradients:
its own output (GRAD_OUT) and/or its inputs (GRAD_IN) -- the "minimum
dependency declaration" of section 3.  ``mirror[v]`` is Alg. 2's m(v): how
many times v's result is recomputed (0: kept).  A node without predecessors
(data) is never recomputed.

Alg. 2 (memory optimized gradient graph construction), as read here:
* a[v] starts as v.  For round k = 1 .. max m, in topological order, every v
  with m(v) >= k gets a new node of v's operator whose predecessors are the
  current a[u] of v's predecessors, and a[v] becomes that node.
* The execution order V' starts with the whole forward graph.  Then, for v in
  reverse topological order, the gradient node g[v] is created: it reads the
  gradient nodes of v's successors, a[v] if v's backward needs its output, and
  a[u] of v's predecessors if it needs its inputs; it produces the gradients
  with respect to v's inputs (sum of their output bytes).  The ancestors of
  g[v] not yet in V', then g[v] itself, are appended in topological order
  (nodes are created in a topological order, so creation order is used).
  Mirror nodes thus run just before the first gradient node that needs them.

Static allocator (section 3, Fig. 3): V' is traversed once; every scheduled
node's output gets a memory tag before execution starts; a liveness counter
per output counts its pending consumers.
* NONE     every output its own tag.
* INPLACE  an INPLACE node whose first input's counter is 1 (it is the last
           pending consumer) and whose tag is at least as large writes its
           output into that input's tag; otherwise a new tag.
* SHARE    INPLACE, and a tag whose output's counter reaches 0 returns to a
           pool; a new output takes the smallest pooled tag that is large
           enough (lowest tag id on ties), else a new tag.
Inputs are released after the node's output is placed (an operator reads its
inputs while it writes its output); an output nobody reads is released right
after its node runs.  Peak = the sum of all tag sizes (the memory allocated
before execution).

Parity: hand-traced two-layer network (tests/golden/graph_small.json);
validity of every tag assignment (no two simultaneously live outputs share a
tag, in-place only on a dead input) and the live-bytes lower bound on random
DAGs; value-level check that every mirror recomputes its original from
equivalent inputs; chain counts (tests/test_oracle_graph.py).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

INPLACE, GRAD_OUT, GRAD_IN = 1, 2, 4
ALLOC_NONE, ALLOC_INPLACE, ALLOC_SHARE = 0, 1, 2
FWD, MIRROR, GRAD = 0, 1, 2


class GraphError(ValueError):
    pass


@dataclass
class Node:
    kind: int                 # FWD, MIRROR or GRAD
    of: int                   # the forward node it derives from
    inputs: List[int]         # ids of the nodes it reads
    bytes: int
    inplace: bool


@dataclass
class GraphPlan:
    nodes: List[Node]
    order: List[int]                   # execution order (node ids)
    tag_of: Dict[int, int] = field(default_factory=dict)   # node id -> tag (-1: no output)
    tag_bytes: List[int] = field(default_factory=list)

    @property
    def peak(self) -> int:
        return sum(self.tag_bytes)

    @property
    def n_mirror(self) -> int:
        return sum(1 for i in self.order if self.nodes[i].kind == MIRROR)


def build(pred: Sequence[Sequence[int]], out_bytes: Sequence[int], flags: Sequence[int],
          mirror: Optional[Sequence[int]] = None) -> GraphPlan:
    """Alg. 2: the gradient graph with mirror nodes and its execution order."""
    n = len(pred)
    if n <= 0 or len(out_bytes) != n or len(flags) != n:
        raise GraphError("a non-empty graph with one size and one flag word per node")
    m = [0] * n if mirror is None else list(mirror)
    if len(m) != n or any(x < 0 for x in m):
        raise GraphError("mirror counts are non-negative, one per node")
    for v in range(n):
        if any(u < 0 or u >= v for u in pred[v]):
            raise GraphError("nodes must be listed in topological order")
        if not pred[v]:
            m[v] = 0  # a graph input is never recomputed
    nodes = [Node(FWD, v, list(pred[v]), int(out_bytes[v]), bool(flags[v] & INPLACE))
             for v in range(n)]
    a = list(range(n))
    for k in range(1, max(m) + 1):
        for v in range(n):
            if k <= m[v]:
                nodes.append(Node(MIRROR, v, [a[u] for u in pred[v]], int(out_bytes[v]),
                                  bool(flags[v] & INPLACE)))
                a[v] = len(nodes) - 1
    succ: List[List[int]] = [[] for _ in range(n)]
    for v in range(n):
        for u in pred[v]:
            if v not in succ[u]:
                succ[u].append(v)
    g = [-1] * n
    order = list(range(n))
    scheduled = set(order)
    for v in range(n - 1, -1, -1):
        ins = [g[s] for s in succ[v]]
        if flags[v] & GRAD_OUT:
            ins.append(a[v])
        if flags[v] & GRAD_IN:
            ins.extend(a[u] for u in pred[v])
        nodes.append(Node(GRAD, v, ins, sum(int(out_bytes[u]) for u in pred[v]),
                          bool(flags[v] & INPLACE)))
        g[v] = len(nodes) - 1
        # ancestors of g[v] not yet scheduled, in creation (topological) order
        need, stack = set(), [g[v]]
        while stack:
            w = stack.pop()
            if w in scheduled or w in need:
                continue
            need.add(w)
            stack.extend(nodes[w].inputs)
        for w in sorted(need):
            order.append(w)
            scheduled.add(w)
    return GraphPlan(nodes, order)


def allocate(plan: GraphPlan, strategy: int) -> GraphPlan:
    """Section 3's static allocation over the execution order (see the header)."""
    if strategy not in (ALLOC_NONE, ALLOC_INPLACE, ALLOC_SHARE):
        raise GraphError("unknown allocation strategy")
    nodes, order = plan.nodes, plan.order
    pos = {w: i for i, w in enumerate(order)}
    count = {w: 0 for w in order}
    for w in order:
        for i in nodes[w].inputs:
            assert pos[i] < pos[w], "an input runs before its reader"
            count[i] += 1
    tag_of: Dict[int, int] = {}
    tag_bytes: List[int] = []
    pool: List[int] = []           # free tags

    def release(i):
        t = tag_of[i]
        if strategy == ALLOC_SHARE and t >= 0:
            pool.append(t)

    for w in order:
        nd = nodes[w]
        tag = -1
        if nd.bytes > 0:
            first = nd.inputs[0] if nd.inputs else -1
            if (strategy != ALLOC_NONE and nd.inplace and first >= 0 and count[first] == 1
                    and tag_of[first] >= 0 and tag_bytes[tag_of[first]] >= nd.bytes):
                tag = tag_of[first]
                count[first] = 0       # consumed by the in-place write: not released
            elif strategy == ALLOC_SHARE:
                fit = [t for t in pool if tag_bytes[t] >= nd.bytes]
                if fit:
                    tag = min(fit, key=lambda t: (tag_bytes[t], t))
                    pool.remove(tag)
            if tag < 0:
                tag = len(tag_bytes)
                tag_bytes.append(nd.bytes)
        tag_of[w] = tag
        for i in nd.inputs:
            if count[i] > 0:
                count[i] -= 1
                if count[i] == 0:
                    release(i)
        if count[w] == 0 and tag >= 0:  # an output nobody reads
            release(w)
    plan.tag_of = tag_of
    plan.tag_bytes = tag_bytes
    return plan


def plan(pred, out_bytes, flags, mirror=None, strategy=ALLOC_SHARE) -> GraphPlan:
    return allocate(build(pred, out_bytes, flags, mirror), strategy)
