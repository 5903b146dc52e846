"""Static check of the bf16 GEMM's LDS synchronisation (no GPU).

The direct loop frees an LDS stage at a bare s_barrier: after it, other
wavefronts' global->LDS loads overwrite the stage the previous slice was read
from.  Every LDS read a wavefront has issued must therefore have returned
before it reaches that barrier.  The compiler may place the MFMAs that consume
a slice's operands (and with them its own wait for the reads) after the next
barrier, so the kernel waits for its LDS reads explicitly.  This test compiles
a few instances of the kernel for gfx950 (dense, forward gather, data-gradient
gather with the transposing reads, weight-gradient gather; four and eight
wavefronts; two and three stages) and walks each one's instructions: at every
s_barrier no LDS read issued since the last lgkmcnt(0) wait may be pending.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

INSTANCES = """
#include "gemm_bf16_kernel.h"
namespace ckpt {
namespace gb {
template __global__ void k_gemm_bf16<64, 64, 2, 2, true, true, __bf16, GEMM_EPI_BF16STATS, GA_FWDT, G_DENSE, true, 0>(Args);
template __global__ void k_gemm_bf16<64, 64, 4, 2, true, true, __bf16, GEMM_EPI_BF16STATS, GA_FWDT, G_DENSE, true, 0>(Args);
template __global__ void k_gemm_bf16<256, 64, 4, 2, true, false, __bf16, GEMM_EPI_BNBWD, GA_DGRADT, GB_WDGRAD, true, 0>(Args);
template __global__ void k_gemm_bf16<128, 128, 2, 2, false, false, __bf16, GEMM_EPI_STORE, G_DENSE, G_DENSE, true, 3>(Args);
template __global__ void k_gemm_bf16<128, 64, 4, 2, false, false, __bf16, GEMM_EPI_STORE, G_DENSE, GB_WGRAD, true, 0>(Args);
template __global__ void k_gemm_bf16<128, 128, 2, 2, true, true, __bf16, GEMM_EPI_ADDMASK, G_DENSE, G_DENSE, true, 0>(Args);
}  // namespace gb
}  // namespace ckpt
"""


def pending_reads_at_barriers(asm: str):
    """{kernel: barriers reached with LDS reads outstanding}, walking each
    kernel's instructions in order (an lgkmcnt(0) wait clears the reads)."""
    bad, kernel, pending = {}, None, 0
    for line in asm.split("\n"):
        m = re.match(r"^(_Z\S+):", line)
        if m:
            kernel, pending = m.group(1), 0
            continue
        if line.startswith(".Lfunc_end"):
            kernel = None
            continue
        tok = line.strip().split()
        if kernel is None or not tok:
            continue
        op = tok[0]
        if op.startswith(("ds_read", "ds_load")):
            pending += 1
        elif op == "s_waitcnt":
            w = re.search(r"lgkmcnt\((\d+)\)", " ".join(tok[1:]))
            if w and int(w.group(1)) == 0:
                pending = 0
        elif op == "s_barrier":
            if pending:
                bad[kernel] = bad.get(kernel, 0) + 1
            pending = 0
    return bad


def test_scan_flags_a_pending_read():
    """The scan itself: a read between the last wait and a barrier is found."""
    asm = "\n".join(["_Zk:", "  ds_read_b128 v[0:3], v4", "  s_waitcnt lgkmcnt(0)", "  s_barrier",
                     "  ds_read_b128 v[0:3], v4", "  s_waitcnt vmcnt(4)", "  s_barrier", ".Lfunc_end0:"])
    assert pending_reads_at_barriers(asm) == {"_Zk": 1}


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None, reason="hipcc not present")
def test_direct_loop_barriers_have_no_pending_lds_reads(tmp_path):
    src = tmp_path / "instances.hip"
    src.write_text(INSTANCES)
    out = tmp_path / "instances.s"
    cmd = [HIPCC if os.path.exists(HIPCC) else "hipcc", "-O3", "-std=c++17",
           "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_1604_06174_amd", "csrc"),
           "-x", "hip", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "--cuda-device-only", "-S", str(src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    asm = out.read_text()
    kernels = re.findall(r"^(_Z\S*k_gemm_bf16\S*):", asm, re.M)
    assert len(kernels) == 6, kernels
    assert sum(1 for l in asm.split("\n") if l.strip().startswith("s_barrier")) > 0
    assert pending_reads_at_barriers(asm) == {}
