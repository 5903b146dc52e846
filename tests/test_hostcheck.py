"""The sanitized host-only build of the library (CPU).

Every library source is compiled for the host side only under
AddressSanitizer and UBSan and linked with a stand-in HIP runtime that checks
kernel launches instead of running them (tests/hostcheck).  The driver fuzzes
the planners, the budget search and the gradient-graph allocator against the
oracle through that build, and dry-runs whole training steps of every net
kind -- the 1000-layer bottleneck ResNet, CIFAR-110, the T = 4096 LSTM, both
MLPs at full size, small nets under every plan, the static-scratch step, the
node-graph step and a recorded step -- on fake device addresses, so that a
host dereference of device memory faults, every kernel's pointers must lie in
the buffers the ABI documents, and the bf16 GEMM's operands must fit them over
their whole extent.
"""
import json
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "hostcheck"))

import build as HB  # noqa: E402


@pytest.fixture(scope="module")
def env():
    if HB.stale():
        HB.build()
    e = dict(os.environ)
    e["LD_PRELOAD"] = HB.runtime()
    e["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    e["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    return e


def _run(env, *args):
    r = subprocess.run([sys.executable, os.path.join(HERE, "hostcheck", "run.py"), *args], env=env,
                       capture_output=True, text=True, timeout=600)
    last = r.stdout.strip().splitlines()[-1] if r.stdout.strip() else "{}"
    try:
        res = json.loads(last)
    except ValueError:
        res = {}
    return r, res


def test_sanitized_dry_run_of_every_step(env):
    r, res = _run(env)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-6000:]
    assert res["checker_errors"] == 0 and not res["failures"]
    assert res["launches"] > 90000 and res["extent_checks"] > 100000


def test_launch_checker_notices_planted_short_buffers(env):
    """A workspace 8 MiB short of its stated size, and a GEMM output one
    element short, are both reported."""
    r, res = _run(env, "--plant")
    assert r.returncode == 1, r.stdout[-2000:] + r.stderr[-4000:]
    assert res["step_errors"] > 0 and res["gemm_errors"] == 1
    assert "in no device allocation" in r.stderr and "spans" in r.stderr
