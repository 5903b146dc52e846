"""Thin ctypes binding of libckpt (include/ckpt.h).

Argument marshalling only: every step of the training path runs in the
library's HIP kernels.  Device buffers are passed as torch tensors (their
``data_ptr()``) or raw integer addresses; the library never allocates device
memory.  Importing this module fails loudly when libckpt.so has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libckpt.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_1604_06174_amd.build`")

# The library links libamdhip64.so.7.  PyTorch ships its own HIP runtime under
# the unversioned name libamdhip64.so; if the library were mapped first, torch
# would load that second copy (and a second HSA runtime) into the process.
# Importing torch first lets the library bind to torch's runtime by soname.
import torch  # noqa: E402,F401  (loads the process's one HIP runtime)

_lib = C.CDLL(LIB_PATH)


def _hip_runtimes():
    try:
        with open("/proc/self/maps") as f:
            return sorted({ln.split()[-1] for ln in f if "libamdhip64.so" in ln})
    except OSError:
        return []


if len(_hip_runtimes()) > 1:
    raise ImportError("two HIP runtimes are mapped into this process: " + ", ".join(_hip_runtimes()))

OK, E_INVALID, E_WORKSPACE, E_MISMATCH, E_HIP, E_UNSUPPORTED = 0, -1, -2, -3, -4, -5
NONE, SQRT, GREEDY, RECURSIVE, USER = 0, 1, 2, 3, 4
FLAG_KEEP_LAST = 1
NET_MLP, NET_RESNET_BASIC, NET_LSTM, NET_RESNET_BOTTLENECK = 1, 2, 3, 4

_u64p = C.POINTER(C.c_uint64)
_i32p = C.POINTER(C.c_int32)


class NetDesc(C.Structure):
    _fields_ = [("kind", C.c_int32), ("batch", C.c_int32), ("depth", C.c_int32),
                ("width", C.c_int32), ("image", C.c_int32), ("n_classes", C.c_int32),
                ("grad_chunk", C.c_int32), ("stage_blocks", C.c_int32 * 4),
                ("expansion", C.c_int32), ("stem_channels", C.c_int32),
                ("drop_bn_relu", C.c_int32), ("reserved", C.c_int32 * 2)]


class Batch(C.Structure):
    _fields_ = [("input", C.c_void_p), ("target", C.c_void_p)]


class StepStats(C.Structure):
    _fields_ = [("unit_forwards", C.c_uint64), ("unit_backwards", C.c_uint64),
                ("kernel_launches", C.c_uint64), ("ckpt_bytes", C.c_uint64),
                ("arena_bytes", C.c_uint64), ("grad_bytes", C.c_uint64)]

    def as_dict(self):
        return {k: int(getattr(self, k)) for k, _ in self._fields_}


def _sig(name, res, args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = args
    return f


_sig("ckpt_last_error", C.c_char_p, [])
_sig("plan_checkpoints", C.c_int, [C.c_int32, _u64p, _u64p, C.c_uint64, C.c_int32, _i32p,
                                   C.c_int32, C.c_int32, C.POINTER(C.c_void_p)])
_sig("plan_info", C.c_int, [C.c_void_p, _i32p, _i32p, _i32p, _u64p, _u64p, _u64p])
_sig("plan_cuts", C.c_int, [C.c_void_p, _i32p, C.c_int32, _i32p])
_sig("plan_serialize", C.c_int, [C.c_void_p, C.POINTER(C.c_uint8), C.c_uint64, _u64p])
_sig("plan_free", None, [C.c_void_p])
_sig("plan_search", C.c_int, [C.c_int32, _u64p, _u64p, _u64p, _u64p, _u64p, C.c_uint64, C.c_uint64,
                              C.c_int32, C.POINTER(C.c_void_p), _u64p, _u64p])
_sig("graph_plan", C.c_int, [C.c_int32, _i32p, _i32p, _u64p, _i32p, _i32p, C.c_int32,
                             C.POINTER(C.c_void_p)])
_sig("graph_plan_info", C.c_int, [C.c_void_p, _i32p, _i32p, _i32p, _u64p])
_sig("graph_plan_schedule", C.c_int, [C.c_void_p, _i32p, _i32p, _i32p, C.c_int32, _i32p])
_sig("graph_plan_blocks", C.c_int, [C.c_void_p, _u64p, C.c_int32, _i32p])
_sig("graph_plan_free", None, [C.c_void_p])
_sig("net_create", C.c_int, [C.POINTER(NetDesc), C.POINTER(C.c_void_p)])
_sig("net_node_graph", C.c_int, [C.c_void_p, _i32p, _i32p, _i32p, _i32p, _u64p, _i32p, C.c_int32,
                                 C.c_int32])
_sig("graph_workspace_bytes", C.c_int, [C.c_void_p, C.c_void_p, _u64p])
_sig("net_destroy", None, [C.c_void_p])
_sig("net_units", C.c_int, [C.c_void_p, _i32p])
_sig("net_unit_sizes", C.c_int, [C.c_void_p, _u64p, _u64p, _u64p])
_sig("net_layer_sizes", C.c_int, [C.c_void_p, _u64p, _u64p])
_sig("net_grad_bytes", C.c_int, [C.c_void_p, _u64p, _u64p])
_sig("net_param_bytes", C.c_int, [C.c_void_p, _u64p])
_sig("net_param_count", C.c_int, [C.c_void_p, _i32p])
_sig("net_param_info", C.c_int, [C.c_void_p, C.c_int32, C.c_char_p, C.c_int32, _u64p, _u64p])
_sig("plan_accounting", C.c_int, [C.c_void_p, C.c_void_p, _u64p, _u64p, _u64p, _u64p])
_sig("net_workspace_bytes", C.c_int, [C.c_void_p, C.c_void_p, _u64p])
_sig("net_set_side_stream", C.c_int, [C.c_void_p, C.c_int32])
_sig("net_timing_enable", C.c_int, [C.c_void_p, C.c_int32])
_sig("net_timing_roofline", C.c_int, [C.c_void_p, C.c_double, C.c_double, C.POINTER(C.c_double),
                                      C.POINTER(C.c_double), C.POINTER(C.c_double)])
_sig("net_timing_read", C.c_int, [C.c_void_p, _u64p, C.POINTER(C.c_double), C.POINTER(C.c_double),
                                  C.POINTER(C.c_double), C.c_char_p, C.c_int32])
_sig("train_step", C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.POINTER(Batch), C.c_void_p,
                             C.c_void_p, C.c_uint64, C.c_void_p, C.POINTER(C.c_float),
                             C.POINTER(C.c_float), _u64p, C.POINTER(StepStats)])
_sig("step_graph_create", C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.POINTER(Batch),
                                    C.c_void_p, C.c_void_p, C.c_uint64, C.c_void_p,
                                    C.POINTER(C.c_float), C.POINTER(C.c_void_p),
                                    C.POINTER(StepStats)])
_sig("train_step_static", C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.POINTER(Batch), C.c_void_p,
                                    C.c_void_p, C.POINTER(C.c_float), C.POINTER(C.c_float), _u64p,
                                    C.POINTER(StepStats)])
STATIC_SCRATCH_BYTES = 64 << 20
_sig("step_graph_launch", C.c_int, [C.c_void_p, C.c_void_p])
_sig("step_graph_free", None, [C.c_void_p])
_sig("train_step_graph", C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.POINTER(Batch), C.c_void_p,
                                   C.c_void_p, C.c_uint64, C.c_void_p, C.POINTER(C.c_float),
                                   C.POINTER(C.c_float), _u64p, C.POINTER(StepStats)])


class ConvGeo(C.Structure):
    _fields_ = [(k, C.c_int32) for k in ("n", "h", "w", "ci", "ho", "wo", "co", "r", "s", "p")]


_vp = C.c_void_p
_sig("op_gemm_bf16_blocks", C.c_int, [C.c_int32, C.c_int32, _i32p, _i32p])
_sig("op_gemm_bf16", C.c_int, [C.c_int32, C.c_int32, C.c_int32, _vp, C.c_int32, C.c_int32, C.c_int32,
                               _vp, C.c_int32, C.c_int32, _vp, C.c_int32, C.c_int32, _vp, C.c_int32,
                               _vp, C.c_int32, _vp, _vp, _vp, _vp, _vp, _vp])
_sig("op_sum_partials", C.c_int, [_vp, C.c_int32, C.c_int64, _vp, _vp])
_sig("op_conv_bf16_fwd", C.c_int, [C.POINTER(ConvGeo), _vp, _vp, _vp, _vp, _vp])
_sig("op_conv_bf16_dgrad", C.c_int, [C.POINTER(ConvGeo), _vp, _vp, _vp, C.c_int32, _vp, _vp, _vp,
                                     _vp, _vp, _vp])
_sig("op_conv_bf16_wgrad", C.c_int, [C.POINTER(ConvGeo), _vp, _vp, _vp, C.c_int32, _vp, _vp])
_sig("op_bn_finalize", C.c_int, [C.c_int32, _vp, C.c_int32, C.c_int32, C.c_int64, _vp, _vp, _vp,
                                 C.c_int32, _vp])
_sig("op_bnb_partial_blocks", C.c_int, [C.c_int64, C.c_int32, _i32p])
_sig("op_bnb_apply", C.c_int, [C.c_int32, C.c_int64, C.c_int32, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                               _vp, _vp, _vp])
_sig("op_bnb_backward", C.c_int, [C.c_int64, C.c_int32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                  _vp, _vp])
_sig("op_bnb_backward_apply", C.c_int, [C.c_int64, C.c_int32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp])
_sig("op_im2col7", C.c_int, [C.c_int32] * 6 + [_vp, _vp, _vp])
_sig("op_maxpool", C.c_int, [C.c_int32] * 7 + [_vp, _vp, _vp, _vp, _vp, _vp])

EPI_STORE, EPI_ADD, EPI_BF16STATS, EPI_ADDMASK, EPI_BNBWD = 0, 1, 3, 4, 6
BNB_RES_NONE, BNB_RES_ID, BNB_RES_BN = 0, 1, 2

EXPORTED = ["op_gemm_bf16_blocks", "op_gemm_bf16", "op_sum_partials", "op_conv_bf16_fwd",
            "op_conv_bf16_dgrad", "op_conv_bf16_wgrad", "op_bn_finalize", "op_bnb_partial_blocks",
            "op_bnb_apply", "op_bnb_backward", "op_bnb_backward_apply", "op_im2col7", "op_maxpool",
            "ckpt_last_error", "plan_checkpoints", "plan_info", "plan_cuts", "plan_serialize",
            "plan_free", "plan_search", "graph_plan", "graph_plan_info", "graph_plan_schedule",
            "graph_plan_blocks", "graph_plan_free", "net_node_graph", "graph_workspace_bytes",
            "train_step_graph", "net_create", "net_destroy", "net_units", "net_unit_sizes",
            "net_layer_sizes", "net_grad_bytes", "net_param_bytes", "net_param_count", "net_param_info",
            "plan_accounting", "net_workspace_bytes", "net_set_side_stream", "net_timing_enable", "net_timing_read", "net_timing_roofline",
            "train_step", "train_step_static", "step_graph_create", "step_graph_launch", "step_graph_free"]


class CkptError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


def _check(rc: int):
    if rc != OK:
        raise CkptError(rc, _lib.ckpt_last_error().decode())


def _u64arr(vals: Sequence[int]):
    return (C.c_uint64 * max(1, len(vals)))(*[int(v) for v in vals])


def _addr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


# ---------------------------------------------------------------- plans --
class Plan:
    """Owner of a library plan object."""

    def __init__(self, handle: int):
        self._h = C.c_void_p(handle)

    @property
    def handle(self):
        return self._h

    def info(self) -> Dict[str, int]:
        mode, n, nc = C.c_int32(), C.c_int32(), C.c_int32()
        x, y, ex = C.c_uint64(), C.c_uint64(), C.c_uint64()
        _check(_lib.plan_info(self._h, C.byref(mode), C.byref(n), C.byref(nc), C.byref(x),
                              C.byref(y), C.byref(ex)))
        return dict(mode=mode.value, n=n.value, n_cuts=nc.value, x=x.value, y=y.value,
                    extra_unit_forwards=ex.value)

    def cuts(self) -> List[int]:
        nc = C.c_int32()
        _check(_lib.plan_cuts(self._h, None, 0, C.byref(nc)))
        buf = (C.c_int32 * max(1, nc.value))()
        _check(_lib.plan_cuts(self._h, buf, nc.value, C.byref(nc)))
        return list(buf[:nc.value])

    def serialize(self) -> bytes:
        ln = C.c_uint64()
        _check(_lib.plan_serialize(self._h, None, 0, C.byref(ln)))
        buf = (C.c_uint8 * ln.value)()
        _check(_lib.plan_serialize(self._h, buf, ln.value, C.byref(ln)))
        return bytes(buf)

    def __del__(self):
        if getattr(self, "_h", None) is not None and self._h.value and _lib is not None:
            _lib.plan_free(self._h)
            self._h = None


def plan_checkpoints(layer_bytes: Sequence[int], cut_bytes: Sequence[int], budget: int, mode: int,
                     user_cuts: Optional[Sequence[int]] = None, flags: int = 0,
                     n_layers: Optional[int] = None) -> Plan:
    n = len(layer_bytes) if n_layers is None else n_layers
    uc = list(user_cuts or [])
    ucarr = (C.c_int32 * max(1, len(uc)))(*uc)
    h = C.c_void_p()
    _check(_lib.plan_checkpoints(n, _u64arr(layer_bytes), _u64arr(cut_bytes), int(budget), mode,
                                 ucarr if user_cuts is not None else None, len(uc), flags,
                                 C.byref(h)))
    return Plan(h.value)


# --------------------------------------------------------------- graphs --
NODE_INPLACE, NODE_GRAD_OUT, NODE_GRAD_IN = 1, 2, 4
ALLOC_NONE, ALLOC_INPLACE, ALLOC_SHARE = 0, 1, 2
GNODE_FORWARD, GNODE_MIRROR, GNODE_GRAD = 0, 1, 2


class GraphPlan:
    """Owner of a library gradient-graph plan (Alg. 2 + the section-3 allocator)."""

    def __init__(self, handle: int):
        self._h = C.c_void_p(handle)

    def info(self) -> Dict[str, int]:
        ne, nm, nb, pk = C.c_int32(), C.c_int32(), C.c_int32(), C.c_uint64()
        _check(_lib.graph_plan_info(self._h, C.byref(ne), C.byref(nm), C.byref(nb), C.byref(pk)))
        return dict(n_exec=ne.value, n_mirror=nm.value, n_blocks=nb.value, peak=pk.value)

    def schedule(self):
        """[(kind, forward node, memory block)] in execution order."""
        n = C.c_int32()
        _check(_lib.graph_plan_schedule(self._h, None, None, None, 0, C.byref(n)))
        k, o, b = [(C.c_int32 * max(1, n.value))() for _ in range(3)]
        _check(_lib.graph_plan_schedule(self._h, k, o, b, n.value, C.byref(n)))
        return list(zip(k[:n.value], o[:n.value], b[:n.value]))

    def blocks(self) -> List[int]:
        n = C.c_int32()
        _check(_lib.graph_plan_blocks(self._h, None, 0, C.byref(n)))
        buf = (C.c_uint64 * max(1, n.value))()
        _check(_lib.graph_plan_blocks(self._h, buf, n.value, C.byref(n)))
        return list(buf[:n.value])

    def __del__(self):
        if getattr(self, "_h", None) is not None and self._h.value and _lib is not None:
            _lib.graph_plan_free(self._h)
            self._h = None


def graph_plan(pred: Sequence[Sequence[int]], out_bytes: Sequence[int], flags: Sequence[int],
               mirror: Optional[Sequence[int]] = None, strategy: int = ALLOC_SHARE,
               n_nodes: Optional[int] = None) -> GraphPlan:
    n = len(pred) if n_nodes is None else n_nodes
    ptr = [0]
    idx: List[int] = []
    for p in pred:
        idx.extend(int(u) for u in p)
        ptr.append(len(idx))
    ptr_a = (C.c_int32 * len(ptr))(*ptr)
    idx_a = (C.c_int32 * max(1, len(idx)))(*idx)
    fl = (C.c_int32 * max(1, len(flags)))(*[int(f) for f in flags])
    mi = None if mirror is None else (C.c_int32 * max(1, len(mirror)))(*[int(m) for m in mirror])
    h = C.c_void_p()
    _check(_lib.graph_plan(n, ptr_a, idx_a, _u64arr(out_bytes), fl, mi, strategy, C.byref(h)))
    return GraphPlan(h.value)


# ----------------------------------------------------------------- nets --
class Net:
    """Owner of a library net object (host descriptor)."""

    def __init__(self, kind: int, batch: int, depth: int, width: int, image: int = 0,
                 n_classes: int = 0, grad_chunk: int = 0, stage_blocks: Sequence[int] = (),
                 expansion: int = 0, stem_channels: int = 0, drop_bn_relu: int = 0):
        sb = list(stage_blocks) + [0] * (4 - len(stage_blocks))
        if len(sb) != 4:
            raise CkptError(E_INVALID, "stage_blocks: at most 4 stages")
        d = NetDesc(kind, batch, depth, width, image, n_classes, grad_chunk,
                    (C.c_int32 * 4)(*sb), expansion, stem_channels, drop_bn_relu)
        h = C.c_void_p()
        _check(_lib.net_create(C.byref(d), C.byref(h)))
        self._h = h

    @property
    def handle(self):
        return self._h

    @property
    def n(self) -> int:
        v = C.c_int32()
        _check(_lib.net_units(self._h, C.byref(v)))
        return v.value

    def unit_sizes(self) -> Tuple[List[int], List[int], List[int]]:
        n = self.n
        b, a, q = (C.c_uint64 * (n + 1))(), (C.c_uint64 * n)(), (C.c_uint64 * n)()
        _check(_lib.net_unit_sizes(self._h, b, a, q))
        return list(b), list(a), list(q)

    def layer_sizes(self) -> Tuple[List[int], List[int]]:
        n = self.n
        lb, cb = (C.c_uint64 * n)(), (C.c_uint64 * n)()
        _check(_lib.net_layer_sizes(self._h, lb, cb))
        return list(lb), list(cb)

    def grad_bytes(self) -> Tuple[int, int]:
        slot, extra = C.c_uint64(), C.c_uint64()
        _check(_lib.net_grad_bytes(self._h, C.byref(slot), C.byref(extra)))
        return slot.value, extra.value

    def search_plan(self, flags: int = 0) -> Tuple["Plan", int, int]:
        """Appendix A's budget search over this net's layout tables."""
        lb, cb = self.layer_sizes()
        b, a, q = self.unit_sizes()
        slot, extra = self.grad_bytes()
        return plan_search(lb, cb, b, a, q, slot, extra, flags)

    def param_bytes(self) -> int:
        v = C.c_uint64()
        _check(_lib.net_param_bytes(self._h, C.byref(v)))
        return v.value

    def param_layout(self) -> List[Tuple[str, int, int]]:
        cnt = C.c_int32()
        _check(_lib.net_param_count(self._h, C.byref(cnt)))
        out = []
        name = C.create_string_buffer(128)
        off, numel = C.c_uint64(), C.c_uint64()
        for k in range(cnt.value):
            _check(_lib.net_param_info(self._h, k, name, 128, C.byref(off), C.byref(numel)))
            out.append((name.value.decode(), off.value, numel.value))
        return out

    def accounting(self, plan: Plan) -> Dict[str, int]:
        ck, ar, gr, pk = C.c_uint64(), C.c_uint64(), C.c_uint64(), C.c_uint64()
        _check(_lib.plan_accounting(self._h, plan.handle, C.byref(ck), C.byref(ar), C.byref(gr),
                                    C.byref(pk)))
        return dict(ckpt=ck.value, arena=ar.value, grad=gr.value, peak=pk.value)

    def workspace_bytes(self, plan: Plan) -> int:
        v = C.c_uint64()
        _check(_lib.net_workspace_bytes(self._h, plan.handle, C.byref(v)))
        return v.value

    def node_graph(self) -> Dict:
        """The net's operator-level graph: pred lists, bytes and flags."""
        n, e = C.c_int32(), C.c_int32()
        _check(_lib.net_node_graph(self._h, C.byref(n), C.byref(e), None, None, None, None, 0, 0))
        ptr = (C.c_int32 * (n.value + 1))()
        idx = (C.c_int32 * max(1, e.value))()
        by = (C.c_uint64 * n.value)()
        fl = (C.c_int32 * n.value)()
        _check(_lib.net_node_graph(self._h, C.byref(n), C.byref(e), ptr, idx, by, fl, n.value, e.value))
        pred = [list(idx[ptr[v]:ptr[v + 1]]) for v in range(n.value)]
        return dict(pred=pred, bytes=list(by), flags=list(fl))

    def graph_workspace_bytes(self, plan: "GraphPlan") -> int:
        v = C.c_uint64()
        _check(_lib.graph_workspace_bytes(self._h, plan._h, C.byref(v)))
        return v.value

    def set_side_stream(self, on: bool = True):
        """Let (True) or stop (False) the net run its units' weight gradients
        on a second stream beside the input gradients (same bits either way)."""
        _check(_lib.net_set_side_stream(self._h, 1 if on else 0))

    def timing_enable(self, on: bool = True):
        _check(_lib.net_timing_enable(self._h, 1 if on else 0))

    def timing_read(self) -> Dict:
        n = C.c_uint64()
        ms, fl, by = C.c_double(), C.c_double(), C.c_double()
        name = C.create_string_buffer(64)
        _check(_lib.net_timing_read(self._h, C.byref(n), C.byref(ms), C.byref(fl), C.byref(by),
                                    name, 64))
        return dict(launches=n.value, ms=ms.value, flops=fl.value, bytes=by.value,
                    kernel=name.value.decode())

    def timing_roofline(self, peak_flops: float, peak_bytes_per_s: float) -> Dict:
        r, k, b = C.c_double(), C.c_double(), C.c_double()
        _check(_lib.net_timing_roofline(self._h, float(peak_flops), float(peak_bytes_per_s), C.byref(r),
                                        C.byref(k), C.byref(b)))
        return dict(roofline_ms=r.value, kernel_ms=k.value, busy_ms=b.value)

    def __del__(self):
        if getattr(self, "_h", None) is not None and self._h.value and _lib is not None:
            _lib.net_destroy(self._h)
            self._h = None


def plan_search(layer_bytes: Sequence[int], cut_bytes: Sequence[int], b: Sequence[int],
                a: Sequence[int], q: Sequence[int], grad_slot: int = 0, grad_extra: int = 0,
                flags: int = 0) -> Tuple["Plan", int, int]:
    """Appendix A's budget search; returns (GREEDY plan, chosen budget, exact peak)."""
    n = len(layer_bytes)
    arr = lambda v, k: (C.c_uint64 * max(k, 1))(*[int(x) for x in v])
    h = C.c_void_p()
    bud, pk = C.c_uint64(), C.c_uint64()
    _check(_lib.plan_search(n, arr(layer_bytes, n), arr(cut_bytes, n), arr(b, n + 1), arr(a, n),
                            arr(q, n), int(grad_slot), int(grad_extra), flags, C.byref(h),
                            C.byref(bud), C.byref(pk)))
    return Plan(h.value), bud.value, pk.value


def net_create(kind: int, batch: int, depth: int, width: int, image: int = 0,
               n_classes: int = 0, grad_chunk: int = 0, stage_blocks: Sequence[int] = (),
               expansion: int = 0, stem_channels: int = 0, drop_bn_relu: int = 0) -> Net:
    return Net(kind, batch, depth, width, image, n_classes, grad_chunk, stage_blocks, expansion,
               stem_channels, drop_bn_relu)


def train_step_graph(net: Net, params, grads, batch_input, batch_target, plan: GraphPlan, workspace,
                     workspace_bytes: int, stream=None, loss_dev=None, want_loss: bool = True):
    """One step over the net's node graph in a graph plan's order and memory
    blocks; returns (loss or None, planned bytes, stats dict)."""
    b = Batch(_addr(batch_input), _addr(batch_target))
    loss = C.c_float()
    peak = C.c_uint64()
    st = StepStats()
    s = None
    if stream is not None:
        s = stream if isinstance(stream, int) else int(stream.cuda_stream)
    ld = _addr(loss_dev)
    _check(_lib.train_step_graph(net.handle, _addr(params), _addr(grads), C.byref(b), plan._h,
                                 _addr(workspace), int(workspace_bytes), s,
                                 C.cast(C.c_void_p(ld), C.POINTER(C.c_float)) if ld else None,
                                 C.byref(loss) if want_loss else None, C.byref(peak), C.byref(st)))
    return (loss.value if want_loss else None), peak.value, st.as_dict()


def train_step(net: Net, params, grads, batch_input, batch_target, plan: Plan, workspace,
               workspace_bytes: int, stream=None, loss_dev=None, want_loss: bool = True):
    """Run one step; returns (loss or None, peak bytes, stats dict)."""
    b = Batch(_addr(batch_input), _addr(batch_target))
    loss = C.c_float()
    peak = C.c_uint64()
    st = StepStats()
    s = None
    if stream is not None:
        s = stream if isinstance(stream, int) else int(stream.cuda_stream)
    ld = _addr(loss_dev)
    _check(_lib.train_step(net.handle, _addr(params), _addr(grads), C.byref(b), plan.handle,
                           _addr(workspace), int(workspace_bytes), s,
                           C.cast(C.c_void_p(ld), C.POINTER(C.c_float)) if ld else None,
                           C.byref(loss) if want_loss else None, C.byref(peak), C.byref(st)))
    return (loss.value if want_loss else None), peak.value, st.as_dict()


def train_step_static(net: Net, params, grads, batch_input, batch_target, plan: Plan, stream=None,
                      loss_dev=None, want_loss: bool = True):
    """train_step on the library's static per-GPU scratch (no workspace
    argument); returns (loss or None, peak bytes, stats dict)."""
    b = Batch(_addr(batch_input), _addr(batch_target))
    loss = C.c_float()
    peak = C.c_uint64()
    st = StepStats()
    s = None
    if stream is not None:
        s = stream if isinstance(stream, int) else int(stream.cuda_stream)
    ld = _addr(loss_dev)
    _check(_lib.train_step_static(net.handle, _addr(params), _addr(grads), C.byref(b), plan.handle, s,
                                  C.cast(C.c_void_p(ld), C.POINTER(C.c_float)) if ld else None,
                                  C.byref(loss) if want_loss else None, C.byref(peak), C.byref(st)))
    return (loss.value if want_loss else None), peak.value, st.as_dict()


class StepGraph:
    """A train_step recorded as a HIP graph (step_graph_create).  Holds
    references to the buffers the recording uses so they outlive it."""

    def __init__(self, handle: int, keep, stats: Dict):
        self._h = handle
        self._keep = keep
        self.stats = stats

    def launch(self, stream=None):
        s = None
        if stream is not None:
            s = stream if isinstance(stream, int) else int(stream.cuda_stream)
        _check(_lib.step_graph_launch(self._h, s))

    def close(self):
        if self._h:
            _lib.step_graph_free(self._h)
            self._h = None
            self._keep = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def step_graph_create(net: Net, params, grads, batch_input, batch_target, plan: Plan, workspace,
                      workspace_bytes: int, stream, loss_dev=None) -> StepGraph:
    """Record one train_step (loss to loss_dev) on a non-default stream."""
    b = Batch(_addr(batch_input), _addr(batch_target))
    st = StepStats()
    s = stream if isinstance(stream, int) else int(stream.cuda_stream)
    ld = _addr(loss_dev)
    out = C.c_void_p()
    _check(_lib.step_graph_create(net.handle, _addr(params), _addr(grads), C.byref(b), plan.handle,
                                  _addr(workspace), int(workspace_bytes), s,
                                  C.cast(C.c_void_p(ld), C.POINTER(C.c_float)) if ld else None,
                                  C.byref(out), C.byref(st)))
    keep = (net, plan, params, grads, batch_input, batch_target, workspace, loss_dev)
    return StepGraph(out.value, keep, st.as_dict())


# ------------------------------------------------------------ operators --
def _s(stream):
    if stream is None:
        return None
    return stream if isinstance(stream, int) else int(stream.cuda_stream)


def conv_geo(n, h, w, ci, ho, wo, co, r, s, p) -> ConvGeo:
    return ConvGeo(n, h, w, ci, ho, wo, co, r, s, p)


def op_gemm_bf16_blocks(m: int, n: int) -> Tuple[int, int]:
    rb, cb = C.c_int32(), C.c_int32()
    _check(_lib.op_gemm_bf16_blocks(m, n, C.byref(rb), C.byref(cb)))
    return rb.value, cb.value


def op_gemm_bf16(m, n, k, a, lda, ak, b, ldb, bk, c, ldc, epi=EPI_STORE, d=None, ldd=0, bias=None,
                 splits=1, mask=None, cb=None, stats=None, cv=None, bst=None, a_fp32=False,
                 stream=None):
    _check(_lib.op_gemm_bf16(m, n, k, _addr(a), int(a_fp32), lda, int(ak), _addr(b), ldb, int(bk),
                             _addr(c), ldc, epi, _addr(d), ldd, _addr(bias), splits, _addr(mask),
                             _addr(cb), _addr(stats), _addr(cv), _addr(bst), _s(stream)))


def op_sum_partials(part, nb, count, out, stream=None):
    _check(_lib.op_sum_partials(_addr(part), nb, count, _addr(out), _s(stream)))


def op_conv_bf16_fwd(geo, x, w, y, stats, stream=None):
    _check(_lib.op_conv_bf16_fwd(C.byref(geo), _addr(x), _addr(w), _addr(y), _addr(stats), _s(stream)))


def op_conv_bf16_dgrad(geo, dy, w, dx, epi=EPI_STORE, d=None, mask=None, cv=None, bst=None,
                       stats=None, stream=None):
    _check(_lib.op_conv_bf16_dgrad(C.byref(geo), _addr(dy), _addr(w), _addr(dx), epi, _addr(d),
                                   _addr(mask), _addr(cv), _addr(bst), _addr(stats), _s(stream)))


def op_conv_bf16_wgrad(geo, x, dy, part, splits, dw, stream=None):
    _check(_lib.op_conv_bf16_wgrad(C.byref(geo), _addr(x), _addr(dy), _addr(part), splits, _addr(dw),
                                   _s(stream)))


def op_bn_finalize(backward, part, nb, j, m, out, dgamma=None, dbeta=None, channel_major=False,
                   stream=None):
    _check(_lib.op_bn_finalize(int(backward), _addr(part), nb, j, m, _addr(out), _addr(dgamma),
                               _addr(dbeta), int(channel_major), _s(stream)))


def op_bnb_partial_blocks(p: int, j: int) -> int:
    nb = C.c_int32()
    _check(_lib.op_bnb_partial_blocks(p, j, C.byref(nb)))
    return nb.value


def op_bnb_apply(res, p, j, c, st, gamma, beta, x=None, stp=None, gp=None, bp=None, y=None,
                 stream=None):
    _check(_lib.op_bnb_apply(res, p, j, _addr(c), _addr(st), _addr(gamma), _addr(beta), _addr(x),
                             _addr(stp), _addr(gp), _addr(bp), _addr(y), _s(stream)))


def op_bnb_backward(p, j, g, ym, c, st, gamma, part, sums, dgamma, dbeta, d, stream=None):
    _check(_lib.op_bnb_backward(p, j, _addr(g), _addr(ym), _addr(c), _addr(st), _addr(gamma),
                                _addr(part), _addr(sums), _addr(dgamma), _addr(dbeta), _addr(d),
                                _s(stream)))


def op_bnb_backward_apply(p, j, g, ym, c, st, gamma, sums, d, stream=None):
    _check(_lib.op_bnb_backward_apply(p, j, _addr(g), _addr(ym), _addr(c), _addr(st), _addr(gamma),
                                      _addr(sums), _addr(d), _s(stream)))


def op_im2col7(n, h, w, ho, wo, x, col, kp=147, stream=None):
    _check(_lib.op_im2col7(n, h, w, ho, wo, kp, _addr(x), _addr(col), _s(stream)))


def op_maxpool(backward, n, h, w, c, ho, wo, r, out, g=None, y=None, arg=None, stream=None):
    _check(_lib.op_maxpool(int(backward), n, h, w, c, ho, wo, _addr(g), _addr(r), _addr(y), _addr(out),
                           _addr(arg), _s(stream)))
