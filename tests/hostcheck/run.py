"""Driver of the sanitized host-only library (run with the ASan runtime
preloaded; tests/test_hostcheck.py does that).

    LD_PRELOAD=<asan runtime> python tests/hostcheck/run.py [--quick | --plant]
    LD_PRELOAD=<asan runtime> python tests/hostcheck/run.py --gemm-log resnet1000 <file> [--stage-blocks 3,3,3,3 | --seq-len 512]

1. Planner, budget search and gradient-graph fuzzing through the instrumented
   library, each result compared with the oracle (as the CPU ABI tests do on
   the production library).
2. Dry runs of whole training steps: every net kind at its full workload size
   (the 1000-layer bottleneck ResNet under its greedy plan among them) and at
   small sizes under every plan mode, train_step_static, the node-graph steps
   and a recorded step, on fake device buffers sized exactly as the ABI
   documents.  The stand-in HIP runtime checks every kernel launch's pointers
   against those buffers (the bf16 GEMM's over each operand's whole extent).

Exits 0 when every comparison holds and the launch checker counted no error;
AddressSanitizer / UBSan abort the process on a host memory error.  With
--plant it instead runs the 1000-layer ResNet step on a workspace 8 MiB short
of what the library asked for and one bf16 GEMM on an output buffer one
element short, and exits 1 if the checker reports both.
"""
from __future__ import annotations

import ctypes as C
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(HERE))

import synth  # noqa: E402
from oracle import graph as OG, planner as PL, sizes as SZ  # noqa: E402

LIB = C.CDLL(os.path.join(ROOT, "_build", "hostcheck", "libckpt_hostcheck.so"))
u64p, i32p, vp = C.POINTER(C.c_uint64), C.POINTER(C.c_int32), C.c_void_p


class NetDesc(C.Structure):
    _fields_ = [("kind", C.c_int32), ("batch", C.c_int32), ("depth", C.c_int32),
                ("width", C.c_int32), ("image", C.c_int32), ("n_classes", C.c_int32),
                ("grad_chunk", C.c_int32), ("stage_blocks", C.c_int32 * 4),
                ("expansion", C.c_int32), ("stem_channels", C.c_int32),
                ("drop_bn_relu", C.c_int32), ("reserved", C.c_int32 * 2)]


class Batch(C.Structure):
    _fields_ = [("input", vp), ("target", vp)]


class Stats(C.Structure):
    _fields_ = [(k, C.c_uint64) for k in ("unit_forwards", "unit_backwards", "kernel_launches",
                                          "ckpt_bytes", "arena_bytes", "grad_bytes")]


def sig(name, res, args):
    f = getattr(LIB, name)
    f.restype, f.argtypes = res, args


sig("ckpt_last_error", C.c_char_p, [])
sig("hc_alloc", C.c_uint64, [C.c_uint64, C.c_char_p])
sig("hc_free_all", None, [])
sig("hc_counters", None, [u64p, u64p, u64p, u64p])
sig("plan_checkpoints", C.c_int, [C.c_int32, u64p, u64p, C.c_uint64, C.c_int32, i32p, C.c_int32,
                                  C.c_int32, C.POINTER(vp)])
sig("plan_serialize", C.c_int, [vp, C.POINTER(C.c_uint8), C.c_uint64, u64p])
sig("plan_free", None, [vp])
sig("plan_search", C.c_int, [C.c_int32, u64p, u64p, u64p, u64p, u64p, C.c_uint64, C.c_uint64,
                             C.c_int32, C.POINTER(vp), u64p, u64p])
sig("graph_plan", C.c_int, [C.c_int32, i32p, i32p, u64p, i32p, i32p, C.c_int32, C.POINTER(vp)])
sig("graph_plan_info", C.c_int, [vp, i32p, i32p, i32p, u64p])
sig("graph_plan_schedule", C.c_int, [vp, i32p, i32p, i32p, C.c_int32, i32p])
sig("graph_plan_free", None, [vp])
sig("net_create", C.c_int, [C.POINTER(NetDesc), C.POINTER(vp)])
sig("net_destroy", None, [vp])
sig("net_units", C.c_int, [vp, i32p])
sig("net_layer_sizes", C.c_int, [vp, u64p, u64p])
sig("net_param_bytes", C.c_int, [vp, u64p])
sig("net_workspace_bytes", C.c_int, [vp, vp, u64p])
sig("net_node_graph", C.c_int, [vp, i32p, i32p, i32p, i32p, u64p, i32p, C.c_int32, C.c_int32])
sig("graph_workspace_bytes", C.c_int, [vp, vp, u64p])
step_args = [vp, vp, vp, C.POINTER(Batch), vp, vp, C.c_uint64, vp, C.POINTER(C.c_float),
             C.POINTER(C.c_float), u64p, C.POINTER(Stats)]
sig("train_step", C.c_int, step_args)
sig("train_step_graph", C.c_int, step_args)
sig("train_step_static", C.c_int, [vp, vp, vp, C.POINTER(Batch), vp, vp, C.POINTER(C.c_float),
                                   C.POINTER(C.c_float), u64p, C.POINTER(Stats)])
sig("step_graph_create", C.c_int, [vp, vp, vp, C.POINTER(Batch), vp, vp, C.c_uint64, vp,
                                   C.POINTER(C.c_float), C.POINTER(vp), C.POINTER(Stats)])
sig("step_graph_launch", C.c_int, [vp, vp])
sig("step_graph_free", None, [vp])
sig("op_gemm_bf16", C.c_int, [C.c_int32, C.c_int32, C.c_int32, vp, C.c_int32, C.c_int32, C.c_int32, vp,
                              C.c_int32, C.c_int32, vp, C.c_int32, C.c_int32, vp, C.c_int32, vp, C.c_int32,
                              vp, vp, vp, vp, vp, vp])

FAILURES = []
# --plant: hand the library buffers shorter than it was told, so the launch
# checker must object (a workspace 8 MiB short of its size, a GEMM output one
# element short)
SHORT = (8 << 20) if "--plant" in sys.argv else 0


def check(cond, what):
    if not cond:
        FAILURES.append(what)
        print("FAIL:", what, flush=True)


def ok(rc, what):
    if rc != 0:
        check(False, f"{what}: rc {rc} ({LIB.ckpt_last_error().decode()})")
    return rc == 0


def arr(t, v):
    v = list(v)
    return (t * max(1, len(v)))(*v)


# ---------------------------------------------------------------- planners --
def lib_plan(n, lb, cb, budget, mode, user=None, flags=0):
    h = vp()
    uc = arr(C.c_int32, user or [])
    rc = LIB.plan_checkpoints(n, arr(C.c_uint64, lb), arr(C.c_uint64, cb), budget, mode, uc,
                              len(user or []), flags, C.byref(h))
    return rc, h


def serialized(h):
    ln = C.c_uint64()
    LIB.plan_serialize(h, None, 0, C.byref(ln))
    buf = (C.c_uint8 * ln.value)()
    LIB.plan_serialize(h, buf, ln.value, C.byref(ln))
    return bytes(buf)


def fuzz_planner(trials):
    rng = np.random.default_rng(11)
    for trial in range(trials):
        n = int(rng.integers(1, 300)) if trial % 10 else int(rng.integers(1000, 5000))
        lb = [int(v) for v in rng.integers(0, 1 << 20, n)]
        cand = rng.random(n) < (1.0 if trial % 3 == 0 else 0.8)
        cb = [int(v) if c else 0 for v, c in zip(rng.integers(1, 1 << 18, n), cand)]
        cb[-1] = 0
        cases = [(PL.SQRT, 0), (PL.SQRT, int(rng.integers(1, 40))), (PL.GREEDY, 0),
                 (PL.GREEDY, int(rng.integers(0, sum(lb) + 2))), (PL.NONE, 0)]
        if all(c > 0 for c in cb[:-1]):
            cases += [(PL.RECURSIVE, 0), (PL.RECURSIVE, int(rng.integers(1, n + 3)))]
        for mode, budget in cases:
            for flags in ((0, PL.FLAG_KEEP_LAST) if mode != PL.RECURSIVE else (0,)):
                rc, h = lib_plan(n, lb, cb, budget, mode, flags=flags)
                if ok(rc, f"plan n={n} mode={mode}"):
                    want = PL.plan(n, lb, cb, budget, mode, flags=flags).serialize()
                    check(serialized(h) == want, f"plan bytes n={n} mode={mode} budget={budget}")
                    LIB.plan_free(h)
        cands = [i for i in range(n - 1) if cb[i] > 0]
        if cands:
            user = sorted(rng.choice(cands, int(rng.integers(0, min(len(cands), 20) + 1)),
                                     replace=False).tolist())
            rc, h = lib_plan(n, lb, cb, 0, PL.USER, user)
            if ok(rc, "user plan"):
                check(serialized(h) == PL.plan(n, lb, cb, 0, PL.USER, user).serialize(), "user plan bytes")
                LIB.plan_free(h)
        # rejected calls: unsorted user cuts, a last unit marked as a candidate
        if len(cands) >= 2:
            rc, _ = lib_plan(n, lb, cb, 0, PL.USER, [cands[1], cands[0]])
            check(rc == -1, "unsorted user cuts rejected")
        bad = list(cb)
        bad[-1] = 1
        rc, _ = lib_plan(n, lb, bad, 0, PL.SQRT)
        check(rc == -1, "candidate last unit rejected")


def fuzz_search(trials):
    rng = np.random.default_rng(12)
    for it in range(trials):
        n = int(rng.integers(1, 60))
        b = [int(v) for v in rng.integers(1, 1 << 20, n + 1)]
        a = [int(v) for v in rng.integers(0, 1 << 22, n)]
        q = [int(v) for v in rng.integers(0, 1 << 20, n)]
        lb = [a[i] + b[i + 1] for i in range(n)]
        cb = [b[i + 1] if rng.random() < 0.85 else 0 for i in range(n - 1)] + [0]
        slot = int(rng.integers(0, 1 << 21)) if it % 3 == 0 else 0
        extra = int(rng.integers(0, 1 << 20)) if it % 5 == 0 else 0
        flags = PL.FLAG_KEEP_LAST if it % 2 else 0
        h, B, pk = vp(), C.c_uint64(), C.c_uint64()
        rc = LIB.plan_search(n, arr(C.c_uint64, lb), arr(C.c_uint64, cb), arr(C.c_uint64, b),
                             arr(C.c_uint64, a), arr(C.c_uint64, q), slot, extra, flags, C.byref(h),
                             C.byref(B), C.byref(pk))
        if ok(rc, "plan_search"):
            op, OB, opk = PL.search(n, lb, cb, b, a, q, slot or None, extra, flags)
            check((B.value, pk.value) == (OB, opk), f"search budget/peak {it}")
            check(serialized(h) == op.serialize(), f"search plan bytes {it}")
            LIB.plan_free(h)


def random_dag(rng, n):
    pred, ob, fl, mi = [], [], [], []
    for v in range(n):
        k = 0 if v == 0 else int(rng.integers(1, min(v, 3) + 1))
        pred.append(sorted(rng.choice(v, k, replace=False).tolist()) if k else [])
        ob.append(int(rng.integers(1, 1 << 16)))
        fl.append(int(rng.integers(0, 8)))
        mi.append(int(rng.integers(0, 3)))
    return pred, ob, fl, mi


def fuzz_graphs(trials):
    rng = np.random.default_rng(13)
    for _ in range(trials):
        pred, ob, fl, mi = random_dag(rng, int(rng.integers(1, 50)))
        ptr = [0]
        for p in pred:
            ptr.append(ptr[-1] + len(p))
        idx = [u for p in pred for u in p]
        for strategy in (0, 1, 2):
            h = vp()
            rc = LIB.graph_plan(len(pred), arr(C.c_int32, ptr), arr(C.c_int32, idx), arr(C.c_uint64, ob),
                                arr(C.c_int32, fl), arr(C.c_int32, mi), strategy, C.byref(h))
            if not ok(rc, "graph_plan"):
                continue
            op = OG.plan(pred, ob, fl, mi, strategy)
            ne, nm, nb, pk = C.c_int32(), C.c_int32(), C.c_int32(), C.c_uint64()
            LIB.graph_plan_info(h, C.byref(ne), C.byref(nm), C.byref(nb), C.byref(pk))
            check((pk.value, nm.value, ne.value) == (op.peak, op.n_mirror, len(op.order)), "graph peak")
            cap = ne.value
            kind, of, blk, cnt = (C.c_int32 * cap)(), (C.c_int32 * cap)(), (C.c_int32 * cap)(), C.c_int32()
            LIB.graph_plan_schedule(h, kind, of, blk, cap, C.byref(cnt))
            want = [(op.nodes[w].kind, op.nodes[w].of, op.tag_of[w]) for w in op.order]
            check(list(zip(kind, of, blk)) == want, "graph schedule")
            LIB.graph_plan_free(h)


# --------------------------------------------------------------- dry runs --
KINDS = {"mlp": 1, "resnet_basic": 2, "lstm": 3, "resnet_bottleneck": 4}


def net_of(cfg):
    k = cfg["kind"]
    d = NetDesc()
    d.kind, d.batch = KINDS[k], cfg["batch"]
    if k == "mlp":
        d.depth, d.width = cfg["depth"], cfg["width"]
    elif k == "resnet_basic":
        d.depth, d.width, d.image, d.n_classes = (cfg["blocks_per_stage"], cfg.get("base", 16),
                                                  cfg.get("image", 32), cfg.get("classes", 10))
        d.drop_bn_relu = int(bool(cfg.get("drop_bn_relu")))
    elif k == "lstm":
        d.depth, d.width, d.image, d.n_classes = cfg["T"], cfg["hidden"], cfg["input"], cfg["vocab"]
        d.grad_chunk = cfg.get("grad_chunk", 0)
    else:
        sb = tuple(cfg["stage_blocks"])
        d.depth, d.width = len(sb), tuple(cfg.get("widths", (64,)))[0]
        d.image, d.n_classes = cfg.get("image", 224), cfg.get("classes", 1000)
        for t, v in enumerate(sb):
            d.stage_blocks[t] = v
        d.expansion, d.stem_channels = cfg.get("expansion", 4), cfg.get("stem_channels", 64)
        d.drop_bn_relu = int(bool(cfg.get("drop_bn_relu")))
    h = vp()
    if not ok(LIB.net_create(C.byref(d), C.byref(h)), f"net_create {cfg}"):
        return None
    return h


def batch_bytes(cfg):
    k, st = cfg["kind"], synth.structure(cfg)
    n_in = int(np.prod(st.input_shape))
    n_t = int(np.prod(st.target_shape))
    el = 2 if k in ("lstm", "resnet_bottleneck") else 4   # bf16 inputs
    return n_in * el, n_t * 4


def counters():
    v = [C.c_uint64() for _ in range(4)]
    LIB.hc_counters(*[C.byref(x) for x in v])
    return [x.value for x in v]


def dry_step(cfg, plans, static=False, graph_step=False, record=False):
    net = net_of(cfg)
    if net is None:
        return
    n = C.c_int32()
    LIB.net_units(net, C.byref(n))
    n = n.value
    lb, cb = (C.c_uint64 * n)(), (C.c_uint64 * n)()
    LIB.net_layer_sizes(net, lb, cb)
    lb, cb = list(lb), list(cb)
    pb = C.c_uint64()
    LIB.net_param_bytes(net, C.byref(pb))
    ib, tb = batch_bytes(cfg)
    name = cfg.get("name", cfg["kind"])
    for mode, budget, flags in plans:
        if budget == "tenth":
            budget = sum(lb) // 10
        rc, plan = lib_plan(n, lb, cb, budget, mode, flags=flags)
        if not ok(rc, f"{name}: plan"):
            continue
        ws = C.c_uint64()
        LIB.net_workspace_bytes(net, plan, C.byref(ws))
        LIB.hc_free_all()
        params = LIB.hc_alloc(pb.value, b"params")
        grads = LIB.hc_alloc(pb.value, b"grads")
        b = Batch(LIB.hc_alloc(ib, b"input"), LIB.hc_alloc(tb, b"target"))
        work = LIB.hc_alloc(ws.value - SHORT, b"workspace")
        loss_dev = LIB.hc_alloc(4, b"loss")
        loss, peak, st = C.c_float(), C.c_uint64(), Stats()
        before = counters()
        ok(LIB.train_step(net, params, grads, C.byref(b), plan, work, ws.value, None,
                          C.cast(C.c_void_p(loss_dev), C.POINTER(C.c_float)), C.byref(loss),
                          C.byref(peak), C.byref(st)), f"{name}: train_step mode {mode}")
        after = counters()
        check(after[0] - before[0] == st.kernel_launches,
              f"{name}: launches seen {after[0] - before[0]} vs reported {st.kernel_launches}")
        print(f"  {name:28s} mode {mode} budget {budget}: {st.kernel_launches} launches, "
              f"{st.unit_forwards} unit forwards, workspace {ws.value} B", flush=True)
        if static:
            if ws.value <= (64 << 20):
                ok(LIB.train_step_static(net, params, grads, C.byref(b), plan, None, None, C.byref(loss),
                                         C.byref(peak), C.byref(st)), f"{name}: train_step_static")
            else:
                rc = LIB.train_step_static(net, params, grads, C.byref(b), plan, None, None, None, None, None)
                check(rc == -2, f"{name}: static step refuses a workspace beyond its scratch")
        if record:
            g = vp()
            if ok(LIB.step_graph_create(net, params, grads, C.byref(b), plan, work, ws.value, 1,
                                        C.cast(C.c_void_p(loss_dev), C.POINTER(C.c_float)), C.byref(g),
                                        None), f"{name}: step_graph_create"):
                ok(LIB.step_graph_launch(g, 1), f"{name}: step_graph_launch")
                LIB.step_graph_free(g)
        LIB.plan_free(plan)
    if graph_step:
        nn, ne = C.c_int32(), C.c_int32()
        LIB.net_node_graph(net, C.byref(nn), C.byref(ne), None, None, None, None, 0, 0)
        ptr, idx = (C.c_int32 * (nn.value + 1))(), (C.c_int32 * max(1, ne.value))()
        by, fl = (C.c_uint64 * nn.value)(), (C.c_int32 * nn.value)()
        LIB.net_node_graph(net, C.byref(nn), C.byref(ne), ptr, idx, by, fl, nn.value, ne.value)
        for strategy in (0, 1, 2):
            mirror = arr(C.c_int32, [1 if 0 < v < nn.value - 1 and v % 3 == 2 else 0
                                     for v in range(nn.value)])
            gp = vp()
            if not ok(LIB.graph_plan(nn.value, ptr, idx, by, fl, mirror, strategy, C.byref(gp)), "graph plan"):
                continue
            ws = C.c_uint64()
            LIB.graph_workspace_bytes(net, gp, C.byref(ws))
            LIB.hc_free_all()
            params, grads = LIB.hc_alloc(pb.value, b"params"), LIB.hc_alloc(pb.value, b"grads")
            b = Batch(LIB.hc_alloc(ib, b"input"), LIB.hc_alloc(tb, b"target"))
            work = LIB.hc_alloc(ws.value, b"workspace")
            loss = C.c_float()
            ok(LIB.train_step_graph(net, params, grads, C.byref(b), gp, work, ws.value, None, None,
                                    C.byref(loss), None, None), f"{name}: train_step_graph")
            LIB.graph_plan_free(gp)
    LIB.net_destroy(net)


ALL = [(PL.NONE, 0, 0), (PL.SQRT, 0, 0), (PL.SQRT, 0, PL.FLAG_KEEP_LAST), (PL.GREEDY, "tenth", 0),
       (PL.RECURSIVE, 0, 0), (PL.RECURSIVE, 2, 0)]


def dry_runs(quick):
    small = [dict(kind="mlp", depth=9, width=72, batch=37, name="mlp small"),
             dict(kind="resnet_basic", blocks_per_stage=2, base=8, batch=3, image=16, classes=7,
                  name="cifar small"),
             dict(kind="resnet_basic", blocks_per_stage=2, base=8, batch=3, image=16, classes=7,
                  drop_bn_relu=1, name="cifar small drop bn-relu"),
             dict(kind="lstm", T=13, batch=8, input=16, hidden=24, vocab=40, grad_chunk=4,
                  name="lstm small"),
             dict(kind="resnet_bottleneck", stage_blocks=(2, 1, 1, 1), widths=(8, 16, 32, 64),
                  stem_channels=16, image=32, batch=2, classes=10, name="bottleneck small"),
             dict(kind="resnet_bottleneck", stage_blocks=(2, 1, 1, 1), widths=(8, 16, 32, 64),
                  stem_channels=16, image=32, batch=2, classes=10, drop_bn_relu=1,
                  name="bottleneck small drop bn-relu")]
    for cfg in small:
        dry_step(cfg, ALL, static=True, graph_step=cfg["kind"] in ("mlp", "resnet_basic"), record=True)
    full = [("resnet1000", [(PL.GREEDY, "tenth", 0), (PL.NONE, 0, 0)]),
            ("resnet1000 drop bn-relu", [(PL.GREEDY, "tenth", 0)]),
            ("cifar110", [(PL.SQRT, 0, 0)]), ("mlp64", [(PL.SQRT, 8, 0)]),
            ("lstm4096", [(PL.SQRT, 64, 0)]), ("mlp1024", [(PL.RECURSIVE, 0, 0)])]
    if quick:
        full = full[:1]
    for name, plans in full:
        cfg = dict(synth.WORKLOADS[name.split()[0]], name=name)
        if name.endswith("drop bn-relu"):
            cfg["drop_bn_relu"] = 1
        dry_step(cfg, plans, static=True, graph_step=name == "cifar110")


def main():
    quick = "--quick" in sys.argv
    if "--gemm-log" in sys.argv:
        # --gemm-log <workload> <file> [--stage-blocks a,b,c,d]: the
        # workload's step (its default plan) with every bf16 GEMM launch
        # written to <file>
        i = sys.argv.index("--gemm-log")
        name, path = sys.argv[i + 1], sys.argv[i + 2]
        os.environ["HC_GEMM_LOG"] = path
        cfg = dict(synth.WORKLOADS[name], name=name)
        if "--seq-len" in sys.argv:
            # a shorter LSTM with the same per-step launches
            cfg["T"] = int(sys.argv[sys.argv.index("--seq-len") + 1])
        if "--stage-blocks" in sys.argv:
            # a shorter bottleneck net with the same launch shapes
            v = sys.argv[sys.argv.index("--stage-blocks") + 1]
            cfg["stage_blocks"] = tuple(int(t) for t in v.split(","))
        plan = {"greedy": (PL.GREEDY, "tenth", 0), "sqrt": (PL.SQRT, int(cfg.get("stride", 0)), 0),
                "recursive": (PL.RECURSIVE, 0, 0)}[cfg["plan"]]
        dry_step(cfg, [plan])
        sys.exit(0 if not FAILURES and counters()[1] == 0 else 1)
    if SHORT:
        # a 1x1-convolution product [6272, 256] whose output buffer is one
        # float short: the GEMM's whole-extent check must see it
        m, n, k = 2 * 56 * 56, 256, 64
        a = LIB.hc_alloc(m * k * 2, b"A")
        b = LIB.hc_alloc(n * k * 2, b"B")
        c = LIB.hc_alloc(m * n * 4 - 4, b"C")
        ok(LIB.op_gemm_bf16(m, n, k, a, 0, k, 1, b, k, 1, c, n, 0, None, 0, None, 1, None, None, None,
                            None, None, None), "op_gemm_bf16")
        gemm_errors = counters()[1]
        dry_step(dict(synth.WORKLOADS["resnet1000"], name="resnet1000 short workspace"),
                 [(PL.GREEDY, "tenth", 0)])
        launches, errors, _, _ = counters()
        print(json.dumps(dict(launches=launches, checker_errors=errors, gemm_errors=gemm_errors,
                              step_errors=errors - gemm_errors)), flush=True)
        sys.exit(1 if gemm_errors and errors > gemm_errors else 0)
    fuzz_planner(60 if quick else 200)
    fuzz_search(60 if quick else 150)
    fuzz_graphs(40 if quick else 100)
    dry_runs(quick)
    launches, errors, ptrs, extents = counters()
    out = dict(launches=launches, checker_errors=errors, pointer_checks=ptrs, extent_checks=extents,
               failures=FAILURES[:20])
    print(json.dumps(out), flush=True)
    sys.exit(0 if not FAILURES and errors == 0 and launches > 0 else 1)


if __name__ == "__main__":
    main()
