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
* CIFAR stem (3 -> C, S x S): a = conv output (4NSSC); q = one [N,S,S,C]
  tensor.
* basic block (Cin -> Cout, output side S): a = conv1 output, relu(bn1)
  output, conv2 output (3 x 4NSSCout); q = two [N,S,S,Cout] tensors.  With
  the "drop bn-relu" layout (section 4.2: keep the convolution outputs,
  recompute batch norm + ReLU) the relu(bn1) output is not kept: a = 2 x
  4NSSCout.
* batch-norm statistics of the CNNs (a mean/rstd pair, 8C bytes per BN of C
  channels): formed by a unit's first forward and read by its re-runs and
  backward, they are held for the whole step: fixed buffers of the layout
  (grad_layout's extra), one pair per BN of every unit, not part of a_i.
* LSTM step (batch B, hidden H, vocabulary V; bf16 GEMM operands): b = h
  (bf16, 2BH) + c (fp32, 4BH); a = activated gates i,f,g,o (fp32, 16BH) +
  the softmax gradient of its head (fp32, 4BV); q = the total hidden-state
  gradient (fp32, 4BH).  The gradient slot holds (dh, dc) in fp32 (2 x 4BH),
  and the weight gradients of the shared parameters are accumulated over
  fixed chunks of C time steps, which needs per-chunk copies of dz (bf16,
  C*B*4H*2), the head gradient (bf16, C*B*V*2) and h_{t-1}, h_t (bf16, 2 x
  C*B*H*2): those chunk buffers are counted with the gradient buffers.

* bottleneck ResNet (bf16 activations; B(m, c) = a bf16 tensor of m pixels x
  c channels, F(m, c) the fp32 one): b_0 = the bf16 image batch.
  - stem (conv7x7/2 output side s, C0 channels, m = N s s): a = conv output
    and ReLU output (2 x B(m, C0)); q = the max-pool input gradient F(m, C0)
    + the BN input gradient B(m, C0); the boundary is the pooled output.
  - bottleneck (width w, output channels Co, mi / mo input / output pixels):
    a = c1, r1 (B(mi, w) each), c2, r2 (B(mo, w) each), c3 (B(mo, Co)),
    [cp (B(mo, Co))]; q = max(B(mo, Co),
    B(mi, w)) + F(mi, w) + B(mo, w) [+ B(mo, Co)].  With the "drop bn-relu"
    layout (section 4.2) r1 and r2 are not kept but formed again in the
    gradient scratch: a loses B(mi, w) + B(mo, w) and q gains them.
  The gradient slot holds the largest fp32 boundary gradient.

``grad_layout`` returns (gradient slot bytes, extra gradient bytes); for the
fp32 feed-forward chains the slot is the largest boundary and there is no
extra.

Parity: the accounting that consumes these tables is pinned in
tests/test_oracle_planner.py, and the tables themselves against the tensors
the oracle's own unit forwards keep (every unit kind, the drop bn-relu layout
included), each counted in the dtype the layout stores it in.
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
            if u.kind == "stem3":
                a.append(t)
                q.append(t)
            else:
                a.append((2 if cfg.get("drop_bn_relu") else 3) * t)
                q.append(2 * t)
            b.append(t)
        return b, a, q
    if k == "resnet_bottleneck":
        N = cfg["batch"]

        def bf(m, c):
            return align(2 * m * c)

        def f32(m, c):
            return align(4 * m * c)

        img = cfg["image"]
        side = (img + 2 * 3 - 7) // 2 + 1
        b.append(bf(N * img * img, 3))
        for u in structure.units:
            if u.kind == "stem7":
                m = N * side * side
                a.append(2 * bf(m, u.cout))
                q.append(f32(m, u.cout) + bf(m, u.cout))
            else:
                mi, mo, w, co = N * u.hin * u.hin, N * u.hout * u.hout, u.width, u.cout
                relus = bf(mi, w) + bf(mo, w)          # r1, r2
                drop = cfg.get("drop_bn_relu")
                aa = bf(mi, w) + bf(mo, w) + bf(mo, co) + (0 if drop else relus)
                qq = max(bf(mo, co), bf(mi, w)) + f32(mi, w) + bf(mo, w) + (relus if drop else 0)
                if u.proj:
                    aa += bf(mo, co)
                    qq += bf(mo, co)
                a.append(aa)
                q.append(qq)
            b.append(bf(N * u.hout * u.hout, u.cout))
        return b, a, q
    if k == "lstm":
        B, H, V, n = cfg["batch"], cfg["hidden"], cfg["vocab"], structure.n
        bb = align(2 * B * H) + align(4 * B * H)
        aa = align(16 * B * H) + align(4 * B * V)
        qq = align(4 * B * H)
        return [bb] * (n + 1), [aa] * n, [qq] * n
    raise NotImplementedError(f"size table for {k}")


LSTM_GRAD_CHUNK = 32


def grad_layout(structure, grad_chunk=None):
    """(gradient slot bytes, extra gradient bytes) of the static layout;
    grad_chunk is the LSTM's weight-gradient chunk (None or 0: the default)."""
    b, _, _ = tables(structure)
    if structure.kind == "lstm":
        cfg = structure.cfg
        B, H, V = cfg["batch"], cfg["hidden"], cfg["vocab"]
        C = grad_chunk or LSTM_GRAD_CHUNK
        slot = 2 * align(4 * B * H)
        extra = align(C * B * 4 * H * 2) + align(C * B * V * 2) + 2 * align(C * B * H * 2)
        return slot, extra
    if structure.kind == "resnet_bottleneck":
        N = structure.cfg["batch"]
        slot = max(align(4 * N * u.hout * u.hout * u.cout) for u in structure.units)
        return slot, bn_stats_bytes(structure)
    if structure.kind == "resnet_basic":
        return max(b[1:]), bn_stats_bytes(structure)
    return max(b[1:]), 0


def bn_stats_bytes(structure) -> int:
    """The CNNs' batch-norm statistics held for the whole step: one aligned
    mean/rstd pair (8 bytes per channel) per batch norm of every unit."""
    tot = 0
    for u in structure.units:
        if u.kind in ("stem3", "stem7"):
            tot += align(8 * u.cout)
        elif u.kind == "basic":
            tot += 2 * align(8 * u.cout)
        elif u.kind == "bottleneck":
            tot += 2 * align(8 * u.width) + (2 if u.proj else 1) * align(8 * u.cout)
    return tot


def layer_and_cut_bytes(structure):
    """The planner's inputs: layer_bytes[i] = a_i + b_{i+1}; cut_bytes[i] = b_{i+1}
    except for the last unit (never a candidate)."""
    b, a, _ = tables(structure)
    n = structure.n
    lb = [a[i] + b[i + 1] for i in range(n)]
    cb = [b[i + 1] for i in range(n - 1)] + [0]
    return lb, cb
