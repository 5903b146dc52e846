"""Device-side set-up of one workload for libckpt: allocation and upload.

Given host arrays (parameters by name, one batch), this allocates the flat
parameter/gradient buffers and the workspace with torch on the GPU, copies the
values in at the offsets the library reports, and calls ``train_step``.
PyTorch is used for device memory and streams only.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from . import ckpt as K



def net_for(cfg: Dict) -> K.Net:
    kind = cfg["kind"]
    if kind == "mlp":
        return K.net_create(K.NET_MLP, cfg["batch"], cfg["depth"], cfg["width"])
    if kind == "resnet_basic":
        return K.net_create(K.NET_RESNET_BASIC, cfg["batch"], cfg["blocks_per_stage"],
                            cfg.get("base", 16), cfg.get("image", 32), cfg.get("classes", 10),
                            drop_bn_relu=int(bool(cfg.get("drop_bn_relu", 0))))
    if kind == "lstm":
        return K.net_create(K.NET_LSTM, cfg["batch"], cfg["T"], cfg["hidden"], cfg["input"],
                            cfg["vocab"], cfg.get("grad_chunk", 0))
    if kind == "resnet_bottleneck":
        sb = tuple(cfg["stage_blocks"])
        widths = tuple(cfg.get("widths", (64, 128, 256, 512)))[:len(sb)]
        w0 = widths[0]
        if any(w != w0 << t for t, w in enumerate(widths)):
            raise K.CkptError(K.E_UNSUPPORTED, "bottleneck widths must double per stage")
        return K.net_create(K.NET_RESNET_BOTTLENECK, cfg["batch"], len(sb), w0,
                            cfg.get("image", 224), cfg.get("classes", 1000), 0, sb,
                            cfg.get("expansion", 4), cfg.get("stem_channels", 64),
                            drop_bn_relu=int(bool(cfg.get("drop_bn_relu", 0))))
    raise K.CkptError(K.E_UNSUPPORTED, f"no GPU network for workload kind {kind!r}")


class GpuStep:
    def __init__(self, cfg: Dict, params: Dict[str, np.ndarray], inp: np.ndarray,
                 target: np.ndarray, device: str = "cuda:0"):
        self.cfg = cfg
        self.device = torch.device(device)
        self.net = net_for(cfg)
        self.layout = self.net.param_layout()
        nbytes = self.net.param_bytes()
        self.params = torch.zeros(nbytes // 4, dtype=torch.float32, device=self.device)
        self.grads = torch.zeros(nbytes // 4, dtype=torch.float32, device=self.device)
        host = np.zeros(nbytes // 4, dtype=np.float32)
        for name, off, numel in self.layout:
            v = np.asarray(params[name], dtype=np.float32).reshape(-1)
            if v.size != numel:
                raise ValueError(f"{name}: {v.size} values for {numel} elements")
            host[off // 4: off // 4 + numel] = v
        self.params.copy_(torch.from_numpy(host))
        self.input = torch.from_numpy(np.ascontiguousarray(inp)).to(self.device)
        if cfg["kind"] in ("lstm", "resnet_bottleneck"):  # consumed as bf16
            self.input = self.input.to(torch.bfloat16).contiguous()
        self.target = torch.from_numpy(np.ascontiguousarray(target)).to(self.device)
        self._ws = None
        self.loss_dev = torch.zeros(1, dtype=torch.float32, device=self.device)

    def plan(self, mode: int, budget: int = 0, user_cuts=None, flags: int = 0) -> K.Plan:
        lb, cb = self.net.layer_sizes()
        return K.plan_checkpoints(lb, cb, budget, mode, user_cuts, flags)

    def workspace(self, plan: K.Plan) -> torch.Tensor:
        need = self.net.workspace_bytes(plan)
        if self._ws is None or self._ws.numel() < need:
            self._ws = None
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self._ws

    def run(self, plan: K.Plan, stream: Optional[torch.cuda.Stream] = None, want_loss: bool = True):
        ws = self.workspace(plan)
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        return K.train_step(self.net, self.params, self.grads, self.input, self.target, plan, ws,
                            ws.numel(), s, self.loss_dev, want_loss)

    def record(self, plan: K.Plan, stream: torch.cuda.Stream) -> K.StepGraph:
        """One step under `plan` recorded as a HIP graph on a non-default stream;
        launching it repeats run(plan) on the same buffers."""
        ws = self.workspace(plan)
        return K.step_graph_create(self.net, self.params, self.grads, self.input, self.target, plan,
                                   ws, ws.numel(), stream, self.loss_dev)

    def graph_plan(self, mirror=None, strategy: int = K.ALLOC_SHARE) -> K.GraphPlan:
        g = self.net.node_graph()
        return K.graph_plan(g["pred"], g["bytes"], g["flags"], mirror, strategy)

    def run_graph(self, plan: K.GraphPlan, stream: Optional[torch.cuda.Stream] = None,
                  want_loss: bool = True):
        need = self.net.graph_workspace_bytes(plan)
        if self._ws is None or self._ws.numel() < need:
            self._ws = None
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        return K.train_step_graph(self.net, self.params, self.grads, self.input, self.target, plan,
                                  self._ws, self._ws.numel(), s, self.loss_dev, want_loss)

    def grads_host(self) -> Dict[str, np.ndarray]:
        g = self.grads.cpu().numpy()
        return {name: g[off // 4: off // 4 + numel].copy() for name, off, numel in self.layout}

    def grads_bytes(self) -> bytes:
        return self.grads.cpu().numpy().tobytes()
