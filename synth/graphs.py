"""Node-granularity forward graphs of the workloads, and mirror-count choices.

Input descriptions only (no arithmetic of the method): the operators of each
network as nodes with their output bytes, their inputs, whether they may run
in place and what their backward reads (the minimum dependency declaration of
section 3), and the mirror counts m(v) of Alg. 2 for the paper's plans:
* ``mirror_none``      m = 0 everywhere (the ordinary gradient graph);
* ``mirror_bn_relu``   m = 1 on batch-norm and ReLU nodes: their results are
                       dropped and recomputed ("drop bn-relu", section 5);
* ``mirror_segments``  m = 1 on every node except the outputs of every s-th
                       block, the graph inputs and the loss (a segmented plan
                       in Alg. 2's terms: m = 1 inside segments, 0 on their
                       outputs).
A graph is a dict: ``pred`` (list of input lists, topological order),
``bytes``, ``flags``, ``op`` (operator names), ``block_out`` (node of each
block's output, in order).
"""
from __future__ import annotations

from typing import Dict, List

INPLACE, GRAD_OUT, GRAD_IN = 1, 2, 4

# operator -> (may run in place, backward reads its output, backward reads its inputs)
OPS = {
    "data": 0,
    "fc": GRAD_IN,                 # y = x W (+b): dW needs x, dx needs W
    "conv": GRAD_IN,
    "bn": INPLACE | GRAD_IN,       # backward needs the normalised input (from x and the stats)
    "relu": INPLACE | GRAD_OUT,    # backward needs the mask, read from the output
    "sigmoid": INPLACE | GRAD_OUT,
    "add": INPLACE,                # backward passes the gradient to both inputs
    "shortcut": 0,                 # option-A subsample + zero channels: shape-only backward
    "pool": 0,                     # average pool: shape-only backward
    "maxpool": GRAD_IN,
    "loss": GRAD_OUT,              # softmax cross-entropy / MSE: reads its output (and labels)
}


class _G:
    def __init__(self):
        self.pred: List[List[int]] = []
        self.bytes: List[int] = []
        self.op: List[str] = []
        self.block_out: List[int] = []

    def add(self, op: str, inputs, nbytes: int) -> int:
        self.pred.append(list(inputs))
        self.bytes.append(int(nbytes))
        self.op.append(op)
        return len(self.op) - 1

    def done(self) -> Dict:
        return dict(pred=self.pred, bytes=self.bytes, flags=[OPS[o] for o in self.op], op=self.op,
                    block_out=self.block_out)


def two_layer(batch: int = 64, d_in: int = 784, hidden: int = 1000, classes: int = 10,
              elem: int = 4) -> Dict:
    """Section 3's example: data -> fullc -> sigmoid -> fullc -> softmax loss."""
    g = _G()
    x = g.add("data", [], batch * d_in * elem)
    h = g.add("fc", [x], batch * hidden * elem)
    s = g.add("sigmoid", [h], batch * hidden * elem)
    o = g.add("fc", [s], batch * classes * elem)
    g.add("loss", [o], batch * classes * elem)
    return g.done()


def mlp(depth: int, width: int, batch: int, elem: int = 4) -> Dict:
    """Residual MLP blocks y = x + relu(x W + b), MSE head."""
    g = _G()
    t = batch * width * elem
    x = g.add("data", [], t)
    for _ in range(depth):
        z = g.add("fc", [x], t)
        r = g.add("relu", [z], t)
        x = g.add("add", [r, x], t)
        g.block_out.append(x)
    g.add("loss", [x], t)
    return g.done()


def resnet_basic(blocks_per_stage: int, base: int, batch: int, image: int, classes: int,
                 elem: int = 4) -> Dict:
    """CIFAR-shaped net: conv3x3-BN-ReLU stem, 3 stages of basic blocks
    (conv-BN-ReLU-conv-BN + shortcut, ReLU; stride 2 and option-A shortcut at
    stage transitions), average pool, FC, softmax loss."""
    g = _G()
    side, c = image, base
    x = g.add("data", [], batch * side * side * 3 * elem)
    x = g.add("conv", [x], batch * side * side * c * elem)
    x = g.add("bn", [x], batch * side * side * c * elem)
    x = g.add("relu", [x], batch * side * side * c * elem)
    g.block_out.append(x)
    for stage in range(3):
        for b in range(blocks_per_stage):
            down = stage > 0 and b == 0
            co = c * 2 if down else c
            so = side // 2 if down else side
            t = batch * so * so * co * elem
            y = g.add("conv", [x], t)
            y = g.add("bn", [y], t)
            y = g.add("relu", [y], t)
            y = g.add("conv", [y], t)
            y = g.add("bn", [y], t)
            sc = g.add("shortcut", [x], t) if down else x
            y = g.add("add", [y, sc], t)
            x = g.add("relu", [y], t)
            g.block_out.append(x)
            c, side = co, so
    p = g.add("pool", [x], batch * c * elem)
    o = g.add("fc", [p], batch * classes * elem)
    g.add("loss", [o], batch * classes * elem)
    return g.done()


def resnet_bottleneck(stage_blocks=(32, 64, 205, 32), batch: int = 32, image: int = 224,
                      classes: int = 1000, widths=(64, 128, 256, 512), expansion: int = 4,
                      stem: int = 64, elem: int = 2) -> Dict:
    """ImageNet-shaped bottleneck net: conv7x7/2-BN-ReLU, max pool 3x3/2, stages
    of 1x1-3x3-1x1 blocks (BN after each conv, ReLU after the first two, the
    stride on the 3x3, a projection 1x1 + BN in each stage's first block), add,
    ReLU; pool, FC, softmax loss."""
    g = _G()
    side = image // 2
    x = g.add("data", [], batch * image * image * 3 * elem)
    x = g.add("conv", [x], batch * side * side * stem * elem)
    x = g.add("bn", [x], batch * side * side * stem * elem)
    x = g.add("relu", [x], batch * side * side * stem * elem)
    side //= 2
    x = g.add("maxpool", [x], batch * side * side * stem * elem)
    g.block_out.append(x)
    cin = stem
    for s, nb in enumerate(stage_blocks):
        w, co = widths[s], widths[s] * expansion
        for b in range(nb):
            stride = 2 if (s > 0 and b == 0) else 1
            so = side // stride
            y = g.add("conv", [x], batch * side * side * w * elem)
            y = g.add("bn", [y], batch * side * side * w * elem)
            y = g.add("relu", [y], batch * side * side * w * elem)
            y = g.add("conv", [y], batch * so * so * w * elem)
            y = g.add("bn", [y], batch * so * so * w * elem)
            y = g.add("relu", [y], batch * so * so * w * elem)
            y = g.add("conv", [y], batch * so * so * co * elem)
            y = g.add("bn", [y], batch * so * so * co * elem)
            if b == 0:
                sc = g.add("conv", [x], batch * so * so * co * elem)
                sc = g.add("bn", [sc], batch * so * so * co * elem)
            else:
                sc = x
            y = g.add("add", [y, sc], batch * so * so * co * elem)
            x = g.add("relu", [y], batch * so * so * co * elem)
            g.block_out.append(x)
            side, cin = so, co
    p = g.add("pool", [x], batch * cin * 4)
    o = g.add("fc", [p], batch * classes * 4)
    g.add("loss", [o], batch * classes * 4)
    return g.done()


def mirror_none(g: Dict) -> List[int]:
    return [0] * len(g["op"])


def mirror_bn_relu(g: Dict) -> List[int]:
    return [1 if o in ("bn", "relu") else 0 for o in g["op"]]


def mirror_segments(g: Dict, every: int) -> List[int]:
    keep = set(g["block_out"][every - 1::every])
    return [0 if (v in keep or not g["pred"][v] or g["op"][v] == "loss") else 1
            for v in range(len(g["op"]))]


def for_workload(cfg: Dict) -> Dict:
    if cfg["kind"] == "mlp":
        return mlp(cfg["depth"], cfg["width"], cfg["batch"])
    if cfg["kind"] == "resnet_basic":
        return resnet_basic(cfg["blocks_per_stage"], cfg["base"], cfg["batch"], cfg["image"],
                            cfg["classes"])
    if cfg["kind"] == "resnet_bottleneck":
        return resnet_bottleneck(tuple(cfg["stage_blocks"]), cfg["batch"], cfg["image"],
                                 cfg["classes"])
    raise ValueError(f"no node graph for {cfg['kind']}")
