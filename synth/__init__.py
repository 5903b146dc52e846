"""Seeded synthetic inputs shaped like the paper's workloads.

This module is shared by the CPU oracle, the GPU parity tests and the benchmark.
It only draws random numbers and lays out the network structure (unit kinds,
channel counts, strides, parameter names and shapes); it contains none of the
method's arithmetic.

Every generator uses ``numpy.random.Generator(PCG64(seed))`` and draws in a
fixed order: inputs, then labels/targets, then parameters unit by unit in the
order listed by the structure (weights before biases).  All floating values are
returned as float32 (the values both sides start from); labels are int32.

Workloads (the paper's experiments, section 5, with the shapes of the
training configurations described there):

* residual MLP chain: y = x + relu(x W + b); x ~ N(0,1), targets ~ N(0,1),
  W ~ N(0, var) with var = 1/(width*depth) read as a variance, b = 0.
* CIFAR-shaped residual CNN: 3->C stem conv3x3 + BN + ReLU, three stages of
  basic blocks (C, 2C, 4C channels, stride-2 transitions), average pool, FC
  head.  Images ~ U(0,1), labels uniform.  Conv weights He-normal
  N(0, 2/fan_in), BN gamma=1, beta=0, FC weights U(+-1/sqrt(fan_in)).
* single-layer LSTM with a per-step softmax head: x_t ~ N(0,1), labels
  uniform over the vocabulary, every parameter U(-1/32, 1/32).
* ImageNet-shaped bottleneck ResNet: conv7x7/2 stem + BN + ReLU + maxpool,
  four stages of bottleneck blocks, average pool, FC head; same init rules as
  the CIFAR network.
"""
from __future__ import annotations

from collections import OrderedDict
from dataclasses import dataclass, field
from typing import Dict, List, Tuple

import numpy as np

__all__ = [
    "WORKLOADS", "make", "mlp_structure", "resnet_basic_structure",
    "lstm_structure", "resnet_bottleneck_structure", "structure",
]


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


# --------------------------------------------------------------------------
# Structures (names, shapes, unit list).  No arithmetic of the method here.
# --------------------------------------------------------------------------

@dataclass
class Unit:
    kind: str                     # "mlp", "stem3", "basic", "stem7", "bottleneck", "lstm"
    cin: int = 0
    cout: int = 0
    width: int = 0                # bottleneck inner width
    stride: int = 1
    hin: int = 0                  # input spatial side
    hout: int = 0                 # output spatial side
    proj: bool = False            # bottleneck projection shortcut
    params: List[Tuple[str, Tuple[int, ...], str]] = field(default_factory=list)


@dataclass
class Structure:
    kind: str
    cfg: Dict
    units: List[Unit]
    head_params: List[Tuple[str, Tuple[int, ...], str]]
    input_shape: Tuple[int, ...]
    target_shape: Tuple[int, ...]
    target_kind: str              # "normal" or "labels"
    n_classes: int = 0

    @property
    def n(self) -> int:
        return len(self.units)

    def param_list(self) -> List[Tuple[str, Tuple[int, ...], str]]:
        out = []
        for u in self.units:
            out.extend(u.params)
        out.extend(self.head_params)
        return out


def mlp_structure(depth: int, width: int, batch: int) -> Structure:
    units = []
    for i in range(depth):
        units.append(Unit("mlp", cin=width, cout=width,
                          params=[(f"u{i}.W", (width, width), "mlp_w"),
                                  (f"u{i}.b", (width,), "zero")]))
    return Structure("mlp", dict(depth=depth, width=width, batch=batch), units, [],
                     (batch, width), (batch, width), "normal")


def resnet_basic_structure(blocks_per_stage: int, base: int, batch: int,
                           image: int = 32, classes: int = 10,
                           drop_bn_relu: bool = False) -> Structure:
    units = [Unit("stem3", cin=3, cout=base, stride=1, hin=image, hout=image,
                  params=[("u0.W", (base, 3, 3, 3), "he"),
                          ("u0.gamma", (base,), "one"), ("u0.beta", (base,), "zero")])]
    cin, side = base, image
    for s in range(3):
        cout = base * (2 ** s)
        for j in range(blocks_per_stage):
            stride = 2 if (s > 0 and j == 0) else 1
            i = len(units)
            hout = side // stride
            units.append(Unit("basic", cin=cin, cout=cout, stride=stride, hin=side, hout=hout,
                              params=[(f"u{i}.W1", (cout, 3, 3, cin), "he"),
                                      (f"u{i}.gamma1", (cout,), "one"),
                                      (f"u{i}.beta1", (cout,), "zero"),
                                      (f"u{i}.W2", (cout, 3, 3, cout), "he"),
                                      (f"u{i}.gamma2", (cout,), "one"),
                                      (f"u{i}.beta2", (cout,), "zero")]))
            cin, side = cout, hout
    head = [("head.W", (cin, classes), "fc_w"), ("head.b", (classes,), "fc_b")]
    return Structure("resnet_basic", dict(blocks_per_stage=blocks_per_stage, base=base,
                                          batch=batch, image=image, classes=classes,
                                          drop_bn_relu=bool(drop_bn_relu)),
                     units, head, (batch, image, image, 3), (batch,), "labels", classes)


def resnet_bottleneck_structure(stage_blocks=(32, 64, 205, 32), batch: int = 32,
                                image: int = 224, classes: int = 1000,
                                widths=(64, 128, 256, 512), expansion: int = 4,
                                stem_channels: int = 64, drop_bn_relu: bool = False) -> Structure:
    side = (image + 2 * 3 - 7) // 2 + 1          # conv7x7/2 pad 3
    pooled = (side + 2 * 1 - 3) // 2 + 1         # maxpool3x3/2 pad 1
    units = [Unit("stem7", cin=3, cout=stem_channels, stride=2, hin=image, hout=pooled,
                  params=[("u0.W", (stem_channels, 7, 7, 3), "he"),
                          ("u0.gamma", (stem_channels,), "one"),
                          ("u0.beta", (stem_channels,), "zero")])]
    cin, side = stem_channels, pooled
    for s, (nb, w) in enumerate(zip(stage_blocks, widths)):
        cout = w * expansion
        for j in range(nb):
            stride = 2 if (s > 0 and j == 0) else 1
            proj = (j == 0)
            i = len(units)
            hout = side // stride
            ps = [(f"u{i}.W1", (w, 1, 1, cin), "he"), (f"u{i}.gamma1", (w,), "one"),
                  (f"u{i}.beta1", (w,), "zero"),
                  (f"u{i}.W2", (w, 3, 3, w), "he"), (f"u{i}.gamma2", (w,), "one"),
                  (f"u{i}.beta2", (w,), "zero"),
                  (f"u{i}.W3", (cout, 1, 1, w), "he"), (f"u{i}.gamma3", (cout,), "one"),
                  (f"u{i}.beta3", (cout,), "zero")]
            if proj:
                ps += [(f"u{i}.Wp", (cout, 1, 1, cin), "he"), (f"u{i}.gammap", (cout,), "one"),
                       (f"u{i}.betap", (cout,), "zero")]
            units.append(Unit("bottleneck", cin=cin, cout=cout, width=w, stride=stride,
                              hin=side, hout=hout, proj=proj, params=ps))
            cin, side = cout, hout
    head = [("head.W", (cin, classes), "fc_w"), ("head.b", (classes,), "fc_b")]
    return Structure("resnet_bottleneck",
                     dict(stage_blocks=tuple(stage_blocks), batch=batch, image=image,
                          classes=classes, widths=tuple(widths), stem_channels=stem_channels,
                          drop_bn_relu=bool(drop_bn_relu)),
                     units, head, (batch, image, image, 3), (batch,), "labels", classes)


def lstm_structure(T: int, batch: int, input_size: int, hidden: int, vocab: int) -> Structure:
    shared = [("W_x", (input_size, 4 * hidden), "lstm"), ("W_h", (hidden, 4 * hidden), "lstm"),
              ("b", (4 * hidden,), "lstm"), ("W_o", (hidden, vocab), "lstm"),
              ("b_o", (vocab,), "lstm")]
    units = [Unit("lstm", cin=input_size, cout=hidden) for _ in range(T)]
    # the parameters are shared by every step; they are listed once, on the head slot
    return Structure("lstm", dict(T=T, batch=batch, input=input_size, hidden=hidden,
                                  vocab=vocab), units, shared,
                     (T, batch, input_size), (T, batch), "labels", vocab)


def structure(cfg: Dict) -> Structure:
    k = cfg["kind"]
    if k == "mlp":
        return mlp_structure(cfg["depth"], cfg["width"], cfg["batch"])
    if k == "resnet_basic":
        return resnet_basic_structure(cfg["blocks_per_stage"], cfg.get("base", 16), cfg["batch"],
                                      cfg.get("image", 32), cfg.get("classes", 10),
                                      cfg.get("drop_bn_relu", False))
    if k == "resnet_bottleneck":
        return resnet_bottleneck_structure(tuple(cfg["stage_blocks"]), cfg["batch"],
                                           cfg.get("image", 224), cfg.get("classes", 1000),
                                           tuple(cfg.get("widths", (64, 128, 256, 512))),
                                           cfg.get("expansion", 4), cfg.get("stem_channels", 64),
                                           cfg.get("drop_bn_relu", False))
    if k == "lstm":
        return lstm_structure(cfg["T"], cfg["batch"], cfg["input"], cfg["hidden"], cfg["vocab"])
    raise ValueError(f"unknown workload kind {k!r}")


# --------------------------------------------------------------------------
# The workloads of the paper's experiments, at full size.
# --------------------------------------------------------------------------

WORKLOADS: Dict[str, Dict] = {
    # 64-block residual MLP, width 256, batch 64, fp32, a checkpoint every 8 blocks
    "mlp64": dict(kind="mlp", depth=64, width=256, batch=64, seed=1001, plan="sqrt", stride=8,
                  dtype="f32"),
    # CIFAR-shaped residual CNN, 3 stages x 18 basic blocks, batch 128, fp32, sqrt schedule
    "cifar110": dict(kind="resnet_basic", blocks_per_stage=18, base=16, batch=128, image=32,
                     classes=10, seed=1002, plan="sqrt", stride=0, dtype="f32"),
    # single-layer LSTM 1024/1024, batch 64, T=4096, 10k vocab, bf16 GEMM, every 64 steps
    "lstm4096": dict(kind="lstm", T=4096, batch=64, input=1024, hidden=1024, vocab=10000,
                     seed=1003, plan="sqrt", stride=64, dtype="bf16"),
    # ImageNet-shaped ~1000-layer bottleneck ResNet, batch 32, bf16, greedy at 10%
    "resnet1000": dict(kind="resnet_bottleneck", stage_blocks=(32, 64, 205, 32), batch=32,
                       image=224, classes=1000, seed=1004, plan="greedy", budget_frac=0.1,
                       dtype="bf16"),
    # recursive schedule: 1024-block MLP, width 1024, batch 256, fp32
    "mlp1024": dict(kind="mlp", depth=1024, width=1024, batch=256, seed=1005, plan="recursive",
                    dtype="f32"),
    # recursive schedule: the LSTM at T=16384
    "lstm16384": dict(kind="lstm", T=16384, batch=64, input=1024, hidden=1024, vocab=10000,
                      seed=1005, plan="recursive", dtype="bf16"),
}


def _draw(rng: np.random.Generator, init: str, shape, cfg: Dict) -> np.ndarray:
    if init == "zero":
        return np.zeros(shape, np.float32)
    if init == "one":
        return np.ones(shape, np.float32)
    if init == "mlp_w":
        var = cfg.get("w_var", 1.0 / (cfg["width"] * cfg["depth"]))
        return rng.normal(0.0, np.sqrt(var), size=shape).astype(np.float32)
    if init == "he":
        fan_in = int(np.prod(shape[1:]))
        return rng.normal(0.0, np.sqrt(2.0 / fan_in), size=shape).astype(np.float32)
    if init == "fc_w":
        bound = 1.0 / np.sqrt(shape[0])
        return rng.uniform(-bound, bound, size=shape).astype(np.float32)
    if init == "fc_b":
        # fan_in is the FC input width, carried in the config by the caller
        bound = 1.0 / np.sqrt(cfg["_fc_in"])
        return rng.uniform(-bound, bound, size=shape).astype(np.float32)
    if init == "lstm":
        return rng.uniform(-1.0 / 32, 1.0 / 32, size=shape).astype(np.float32)
    raise ValueError(init)


def make(cfg: Dict, seed: int | None = None) -> Dict:
    """Draw one batch and one parameter set for workload ``cfg``.

    Returns ``{"structure", "input", "target", "params"}`` where params is an
    ordered name -> float32 array mapping in structure order.
    """
    st = structure(cfg)
    rng = _rng(cfg.get("seed", 0) if seed is None else seed)
    cfg2 = dict(cfg)
    if st.head_params and st.kind != "lstm":
        cfg2["_fc_in"] = st.head_params[0][1][0]
    # inputs
    if st.kind == "mlp" or st.kind == "lstm":
        x = rng.standard_normal(size=st.input_shape, dtype=np.float32)
    else:
        x = rng.random(size=st.input_shape, dtype=np.float32)
    # targets / labels
    if st.target_kind == "normal":
        t = rng.standard_normal(size=st.target_shape, dtype=np.float32)
    else:
        t = rng.integers(0, st.n_classes, size=st.target_shape, dtype=np.int64).astype(np.int32)
    params = OrderedDict()
    for name, shape, init in st.param_list():
        params[name] = _draw(rng, init, shape, cfg2)
    return {"structure": st, "input": x, "target": t, "params": params}
