"""Per-launch-kind table of the bf16 GEMM family from a rocprofv3 kernel trace.

    python -m paper_1604_06174_amd.profile_table <run_kernel_trace.csv> <gemm launch log>
    python -m paper_1604_06174_amd.profile_table --counters <gemm launch log> <short-step log> \
        <fetch factor> <write factor> <run_counter_collection.csv> ...

The launch log lists every bf16 GEMM launch of one training step with its
shape (tests/hostcheck/run.py --gemm-log <workload> <file> writes it from a
host-only dry run of the same step); the trace gives each dispatch's kernel,
grid and duration.  They are joined on (kernel, grid).  Per launch kind:
launches per step, M x N x K, algorithmic flops (2 M N K) and bytes (each
operand read once -- the gathered convolution input as the tensor it is --
and the result written once, split-K partials not counted), the average
duration over every traced dispatch of that kind, and the fraction of the
kind's roofline time max(flops / 2.5 PFLOP/s, bytes / 8 TB/s) that duration
reaches.  The family line weights every kind by its launches per step.

The --others form does the same for every other kernel of the step (batch
norm, element passes, partial sums), per kernel and grid: counter bytes of a
shorter step over the durations in the full step's trace.

The --counters form joins rocprofv3 counter runs (FETCH_SIZE, WRITE_SIZE,
SQ_VALU_MFMA_BUSY_CYCLES) of a shorter step -- a bottleneck net with fewer
blocks per stage, so the same launch kinds -- with that step's launch log in
dispatch order, and weights each kind by its launches in the full step.
"""
from __future__ import annotations

import csv
import re
import sys
from collections import defaultdict

MFMA_BF16 = 2.5e15
HBM = 8.0e12
EPI = {0: "STORE", 1: "ADD", 3: "BF16STATS", 4: "ADDMASK", 6: "BNBWD", 7: "ROWSOFTMAX"}
FORM = {0: "dense", 1: "fwd-gather", 2: "dgrad-gather", 3: "wgrad-gather", 4: "weights", 5: "cat",
        6: "fwd-gather", 7: "dgrad-gather"}


def read_log(path):
    rows = []
    with open(path) as f:
        for ln in f:
            v = ln.split()
            name = v[0]
            gx, gy, gz, M, N, K, kper, epi, ga, gb, H, W, Ho, Wo, R, S, cshift, lda = map(int, v[1:19])
            rb, xr = (int(v[19]), int(v[20])) if len(v) > 20 else (0, 0)
            nbatch = int(v[21]) if len(v) > 21 else 0
            rows.append(dict(name=name, grid=(gx, gy, gz), M=M, N=N, K=K, epi=epi, ga=ga, gb=gb, H=H,
                             W=W, Ho=Ho, Wo=Wo, R=R, S=S, C=(1 << cshift) if cshift > 0 else 0, rb=rb, xr=xr,
                             nbatch=nbatch))
    return rows


def work(r):
    """(flops, bytes) of one launch."""
    M, N, K, C = r["M"], r["N"], r["K"], r["C"]
    if r["ga"] in (1, 6):
        a = (M // (r["Ho"] * r["Wo"])) * r["H"] * r["W"] * C * 2
    elif r["ga"] in (2, 7):
        a = (M // (r["H"] * r["W"])) * r["Ho"] * r["Wo"] * C * 2
    else:
        a = M * K * 2
    if r["gb"] == 3:
        b = (K // (r["Ho"] * r["Wo"])) * r["H"] * r["W"] * C * 2
    else:
        b = N * K * 2
    mn = M * N
    out = {3: 2 * mn, 6: 4 * mn + 2 * 2 * mn, 4: 4 * mn + 4 * mn + 2 * mn, 1: 8 * mn}.get(r["epi"], 4 * mn)
    # a re-run's BF16STATS epilogue also writes the batch-norm output (and
    # reads the shortcut it adds)
    out += 2 * mn * (r.get("rb", 0) + r.get("xr", 0))
    # a batch of products sharing B: A, the result and the flops once per product
    nb = max(r.get("nbatch", 0), 1)
    return 2.0 * M * N * K * nb, float(nb * (a + out) + b)


def prefix(name):
    """(BM, BN, WM, WN, AK, BK, rest): the instance's template arguments from a
    mangled name, or the leading ones from a demangled name (rocprofv3 prints
    some instances demangled, and its demangler garbles the __bf16 type that
    follows BK, so those are told apart by their grid instead)."""
    if name.startswith("_Z"):
        v = name.split("k_gemm_bf16I", 1)[1]
        parts = []
        for tok in v.split("E")[:6]:
            parts.append(tok.replace("Li", "").replace("Lb", ""))
        return tuple(int(x) for x in parts[:4]) + (parts[4] == "1", parts[5] == "1"), name
    inner = name.split("k_gemm_bf16<", 1)[1].split(",")
    nums = [t.strip() for t in inner[:6]]
    return tuple(int(x) for x in nums[:4]) + (nums[4] == "true", nums[5] == "true"), None


def main(trace, log):
    rows = read_log(log)
    durs = defaultdict(list)
    with open(trace) as f:
        for d in csv.DictReader(f):
            if "k_gemm_bf16" not in d["Kernel_Name"]:
                continue
            wg = int(d["Workgroup_Size_X"])
            grid = (int(d["Grid_Size_X"]) // wg, int(d["Grid_Size_Y"]), int(d["Grid_Size_Z"]))
            t = (int(d["End_Timestamp"]) - int(d["Start_Timestamp"])) * 1e-9
            pre, mangled = prefix(d["Kernel_Name"])
            durs[(mangled, grid) if mangled else (pre, grid)].append(t)
    kinds = defaultdict(lambda: dict(n=0))
    for r in rows:
        k = (r["name"], r["grid"])
        e = kinds[k]
        e["n"] += 1
        e["r"] = r
        fl, by = work(r)
        e["fl"] = e.get("fl", 0.0) + fl
        e["by"] = e.get("by", 0.0) + by
    out = []
    tot_t = tot_roof = tot_f = tot_b = 0.0
    missing = 0
    for k, e in kinds.items():
        r = e["r"]
        fl, by = e["fl"] / e["n"], e["by"] / e["n"]  # means over the kind's launches
        ds = durs.get(k) or durs.get((prefix(k[0])[0], k[1]))
        if not ds:
            missing += e["n"]
            continue
        t = sum(ds) / len(ds)
        roof = max(fl / MFMA_BF16, by / HBM)
        bound = "mfma" if fl / MFMA_BF16 >= by / HBM else "hbm"
        out.append((e["n"] * t, r, e["n"], fl, by, t, roof, bound))
        tot_t += e["n"] * t
        tot_roof += e["n"] * roof
        tot_f += e["n"] * fl
        tot_b += e["n"] * by
    out.sort(key=lambda x: -x[0])
    print(f"| share | launches/step | tile x grid | epilogue | A / B | M x N x K | GFLOP | MB | avg us "
          f"| bound | frac of roofline |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")
    for tt, r, n, fl, by, t, roof, bound in out:
        tile = r["name"].split("ILi")[1].split("E")[0].replace("ELi", "x") if "ILi" in r["name"] else "?"
        print(f"| {100 * tt / tot_t:.1f}% | {n} | {tile} {r['grid'][0]}x{r['grid'][1]}x{r['grid'][2]} | "
              f"{EPI.get(r['epi'], r['epi'])} | {FORM[r['ga']]} / {FORM[r['gb']]} | "
              f"{r['M']} x {r['N']} x {r['K']} | {fl / 1e9:.2f} | {by / 1e6:.1f} | {t * 1e6:.2f} | {bound} | "
              f"{roof / t:.3f} |")
    n_all = sum(e["n"] for e in kinds.values())
    print(f"\nfamily: {n_all} launches per step ({missing} without a traced dispatch), "
          f"{tot_t * 1e3:.2f} ms of kernel time per step; algorithmic {tot_f / 1e12:.2f} TFLOP and "
          f"{tot_b / 1e9:.2f} GB per step; roofline time {tot_roof * 1e3:.2f} ms = "
          f"{tot_roof / tot_t:.3f} of the kernel time; {tot_f / tot_t / 1e12:.1f} TFLOP/s "
          f"({tot_f / tot_t / MFMA_BF16:.3f} of bf16 peak), {tot_b / tot_t / 1e9:.0f} GB/s "
          f"({tot_b / tot_t / HBM:.3f} of HBM)")


def counters_per_kind(csv_paths, short_log):
    """Mean counter values per launch kind, from rocprofv3 counter runs of a
    step whose bf16 GEMM launches short_log lists in order.  The last
    len(short_log) k_gemm_bf16 dispatches of each run are that step; each is
    checked against its log line's grid before it is used."""
    rows = read_log(short_log)
    acc = defaultdict(lambda: defaultdict(list))
    for path in csv_paths:
        per = defaultdict(dict)  # dispatch -> counter -> value (summed over dimensions)
        meta = {}
        with open(path) as f:
            for d in csv.DictReader(f):
                if "k_gemm_bf16" not in d["Kernel_Name"]:
                    continue
                did = int(d["Dispatch_Id"])
                per[did][d["Counter_Name"]] = per[did].get(d["Counter_Name"], 0.0) + float(d["Counter_Value"])
                meta[did] = (int(d["Grid_Size"]), int(d["Workgroup_Size"]),
                             int(d["End_Timestamp"]) - int(d["Start_Timestamp"]))
        ids = sorted(per)
        if len(ids) < len(rows):
            raise SystemExit(f"{path}: {len(ids)} GEMM dispatches, the step has {len(rows)}")
        for r, did in zip(rows, ids[-len(rows):]):
            grid, wg, dur = meta[did]
            gx, gy, gz = r["grid"]
            if grid != gx * gy * gz * wg:
                raise SystemExit(f"{path}: dispatch {did} grid {grid} does not match launch {r}")
            k = (r["name"], r["grid"])
            for c, v in per[did].items():
                acc[k][c].append(v)
            acc[k]["_dur"].append(dur * 1e-9)
    return {k: {c: sum(v) / len(v) for c, v in cs.items()} for k, cs in acc.items()}


def counters_main(log, short_log, csv_paths, fetch_factor, write_factor):
    """Per launch kind of `log` (the full step), HBM bytes from FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch, scaled by the copy calibration) and the MFMA
    busy fraction, measured on the shorter step of short_log; the family line
    weights each kind by its launches in `log`."""
    kinds = counters_per_kind(csv_paths, short_log)
    full = defaultdict(lambda: dict(n=0))
    for r in read_log(log):
        e = full[(r["name"], r["grid"])]
        e["n"] += 1
        e["r"] = r
        e["by"] = e.get("by", 0.0) + work(r)[1]
    n_all = n_cov = 0
    tr = alg = busy_w = dur_w = 0.0
    out = []
    for k, e in full.items():
        n_all += e["n"]
        c = kinds.get(k)
        if not c or "FETCH_SIZE" not in c or "WRITE_SIZE" not in c:
            continue
        n_cov += e["n"]
        by = e["by"] / e["n"]  # mean over the kind's launches
        t = c["FETCH_SIZE"] * 1024 * fetch_factor + c["WRITE_SIZE"] * 1024 * write_factor
        tr += e["n"] * t
        alg += e["n"] * by
        mb = c.get("SQ_VALU_MFMA_BUSY_CYCLES")
        if mb is not None:
            busy_w += e["n"] * mb
            dur_w += e["n"] * c["_dur"] * 2.4e9 * 1024
        out.append((e["n"] * t, e["r"], e["n"], by, t, (mb / (c["_dur"] * 2.4e9 * 1024)) if mb is not None else None))
    out.sort(key=lambda x: -x[0])
    print("| launches/step | tile x grid | epilogue | A / B | M x N x K | algorithmic MB | HBM MB (counters) "
          "| HBM / algorithmic | MFMA busy |")
    print("|---|---|---|---|---|---|---|---|---|")
    for _, r, n, by, t, mb in out:
        tile = r["name"].split("ILi")[1].split("E")[0] if "ILi" in r["name"] else "?"
        print(f"| {n} | {tile} {r['grid'][0]}x{r['grid'][1]}x{r['grid'][2]} | {EPI.get(r['epi'], r['epi'])} | "
              f"{FORM[r['ga']]} / {FORM[r['gb']]} | {r['M']} x {r['N']} x {r['K']} | {by / 1e6:.1f} | "
              f"{t / 1e6:.1f} | {t / by:.2f} | {'' if mb is None else f'{mb:.3f}'} |")
    print(f"\nfamily: {n_all} launches per step, {n_cov} of them of a kind measured; HBM traffic per "
          f"launch {tr / max(n_cov, 1):.0f} B (algorithmic {alg / max(n_cov, 1):.0f} B, ratio "
          f"{tr / max(alg, 1):.3f})" + (f"; MFMA busy {busy_w / dur_w:.3f} of the counted kernels' time" if dur_w else ""))
    return tr / max(n_cov, 1), n_cov, n_all


def other_kernels_main(trace, fetch_csv, write_csv, fetch_factor, write_factor, steps, skip="k_gemm_bf16"):
    """HBM bytes per dispatch (calibrated FETCH_SIZE + WRITE_SIZE, means over
    the counter runs' dispatches of each kernel and total grid size) joined
    with the mean duration of the same kernel and grid in a kernel trace of
    the full step: achieved HBM bandwidth per kernel kind, for every kernel
    but the `skip` family.  `steps` = training steps in the trace."""
    def short(name):
        if name.startswith("_Z"):  # a mangled instance: its name and integral template arguments
            m = re.search(r"(k_[a-z0-9_]+)I((?:L[ib]\d+E)+)E", name)
            if m:
                args = re.findall(r"L([ib])(\d+)E", m.group(2))
                return m.group(1) + "<" + ", ".join(
                    ("true" if v == "1" else "false") if t == "b" else v for t, v in args) + ">"
            m = re.search(r"(k_[a-z0-9_]+)", name)
            return m.group(1) if m else name[:60]
        n = name.replace("(anonymous namespace)::", "").replace("void ", "").replace("ckpt::", "")
        return n.split("(")[0][:60]
    cnt = defaultdict(lambda: defaultdict(list))
    for path, ctr, fac in ((fetch_csv, "FETCH_SIZE", fetch_factor), (write_csv, "WRITE_SIZE", write_factor)):
        per = defaultdict(float)
        key = {}
        with open(path) as f:
            for d in csv.DictReader(f):
                if skip in d["Kernel_Name"] or d["Counter_Name"] != ctr:
                    continue
                did = int(d["Dispatch_Id"])
                per[did] += float(d["Counter_Value"]) * 1024 * fac
                key[did] = (short(d["Kernel_Name"]), int(d["Grid_Size"]))
        for did, v in per.items():
            cnt[key[did]][ctr].append(v)
    dur = defaultdict(list)
    with open(trace) as f:
        for d in csv.DictReader(f):
            if skip in d["Kernel_Name"]:
                continue
            g = int(d["Grid_Size_X"]) * int(d["Grid_Size_Y"]) * int(d["Grid_Size_Z"])
            dur[(short(d["Kernel_Name"]), g)].append((int(d["End_Timestamp"]) - int(d["Start_Timestamp"])) * 1e-9)
    rows = []
    for k, ds in dur.items():
        c = cnt.get(k)
        if not c or "FETCH_SIZE" not in c or "WRITE_SIZE" not in c:
            continue
        by = sum(c["FETCH_SIZE"]) / len(c["FETCH_SIZE"]) + sum(c["WRITE_SIZE"]) / len(c["WRITE_SIZE"])
        t = sum(ds) / len(ds)
        rows.append((len(ds) / steps * t, k, len(ds) / steps, by, t))
    rows.sort(key=lambda x: -x[0])
    print("| kernel | threads | per step | ms per step | HBM MB per dispatch | avg us | HBM TB/s | of 8 TB/s |")
    print("|---|---|---|---|---|---|---|---|")
    for tot, (name, g), n, by, t in rows:
        print(f"| `{name}` | {g} | {n:.0f} | {tot * 1e3:.2f} | {by / 1e6:.2f} | {t * 1e6:.2f} | "
              f"{by / t / 1e12:.2f} | {by / t / 8e12:.2f} |")


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--others":
        # --others <kernel trace csv> <fetch csv> <write csv> <fetch factor> <write factor> <steps in trace>
        other_kernels_main(sys.argv[2], sys.argv[3], sys.argv[4], float(sys.argv[5]), float(sys.argv[6]),
                           float(sys.argv[7]))
        sys.exit(0)
    if len(sys.argv) > 1 and sys.argv[1] == "--counters":
        # --counters <full-step log> <short-step log> <fetch factor> <write factor> <csv> [<csv> ...]
        counters_main(sys.argv[2], sys.argv[3], sys.argv[6:], float(sys.argv[4]), float(sys.argv[5]))
    else:
        main(sys.argv[1], sys.argv[2])
