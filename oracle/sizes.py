"""Per-unit byte tables (b_i, a_i, q_i) of the executor's static layout.

TEST INFRASTRUCTURE ONLY (see the package header).

These restate, independently of the library, which tensors the GPU executor
keeps for each unit kind (the paper counts feature maps and gradients of a
static allocation, excluding parameters and operator workspace, section 5.1):

* b_i -- bytes of the boundary tensor x_i (b_0 is the network input).
* a_i -- bytes of unit i's saved internals (what its backward reads besides
         its input and output).
* q_i -- bytes of unit i's gradient scratch.

Every tensor is rounded up to a multiple of 256 bytes.

Unit kinds (fp32 unless stated):
* residual MLP [B, D]: b = 4BD; a = z (4BD); q = relu-masked gradient (4BD).
* CIFAR stem (3 -> C, S x S): a = conv output (4NSSC) + BN mean/rstd (8C);
  q = one [N,S,S,C] tensor.
* basic block (Cin -> Cout, output side S): a = conv1 output, relu(bn1)
  output, conv2 output (3 x 4NSSCout) + two BN mean/rstd pairs (2 x 8Cout);
  q = two [N,S,S,Cout] tensors.

Parity: the accounting that consumes these tables is pinned in
tests/test_oracle_planner.py; the tables themselves are restated layout
("parity unpinned" beyond equality with the library's own tables).
"""
from __future__ import annotations

from typing import List, Tuple


def align(x: int) -> int:
    return (x + 255) // 256 * 256


def tables(structure) -> Tuple[List[int], List[int], List[int]]:
    k = structure.kind
    cfg = structure.cfg
    b: List[int] = []
    a: List[int] = []
    q: List[int] = []
    if k == "mlp":
        t = align(4 * cfg["batch"] * cfg["width"])
        n = structure.n
        return [t] * (n + 1), [t] * n, [t] * n
    if k == "resnet_basic":
        N = cfg["batch"]
        u0 = structure.units[0]
        b.append(align(4 * N * u0.hin * u0.hin * 3))
        for u in structure.units:
            t = align(4 * N * u.hout * u.hout * u.cout)
            st = align(8 * u.cout)
            if u.kind == "stem3":
                a.append(t + st)
                q.append(t)
            else:
                a.append(3 * t + 2 * st)
                q.append(2 * t)
            b.append(t)
        return b, a, q
    raise NotImplementedError(f"size table for {k}")


def layer_and_cut_bytes(structure):
    """The planner's inputs: layer_bytes[i] = a_i + b_{i+1}; cut_bytes[i] = b_{i+1}
    except for the last unit (never a candidate)."""
    b, a, _ = tables(structure)
    n = structure.n
    lb = [a[i] + b[i + 1] for i in range(n)]
    cb = [b[i + 1] for i in range(n - 1)] + [0]
    return lb, cb
