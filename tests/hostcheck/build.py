"""Build the host-only, sanitized libckpt used by the launch checker.

    python tests/hostcheck/build.py

Every library source (paper_1604_06174_amd/csrc/*.cpp, *.hip) is compiled
for the host side only (--offload-host-only: kernels become launch stubs)
with AddressSanitizer and UBSan, and linked with hip_stub.cpp, a stand-in
HIP runtime that checks launches instead of running them, into
_build/hostcheck/libckpt_hostcheck.so.  The ASan runtime is a shared library
(runtime()) that a process loading this one must preload.  Nothing here runs
on or needs a GPU.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_1604_06174_amd", "csrc")
OUT_DIR = os.path.join(ROOT, "_build", "hostcheck")
LIB = os.path.join(OUT_DIR, "libckpt_hostcheck.so")
CLANG = "/opt/rocm/llvm/bin/clang++"
FLAGS = ["-x", "hip", "--offload-host-only", "--offload-arch=gfx950", "-std=c++17", "-O1", "-g",
         "-fPIC", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
         "-I" + os.path.join(ROOT, "include"), "-Wno-c++20-extensions", "-Wno-unused-command-line-argument"]


def runtime() -> str:
    """Path of the shared ASan runtime the library is linked against."""
    r = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                       text=True, check=True)
    return r.stdout.strip()


def sources():
    out = [os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC)) if f.endswith((".cpp", ".hip"))]
    return out + [os.path.join(HERE, "hip_stub.cpp")]


def _inputs():
    hdrs = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")]
    return sources() + hdrs + [os.path.join(ROOT, "include", "ckpt.h"), __file__]


def stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in _inputs())


def _compile(src: str) -> str:
    obj = os.path.join(OUT_DIR, os.path.basename(src) + ".o")
    r = subprocess.run([CLANG] + FLAGS + ["-c", src, "-o", obj], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{r.stderr}")
    return obj


def build(jobs: int = 8) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, sources()))
    # host-only objects still name their (absent) device code blobs: define
    # each as an empty array so the registration stubs get a valid address
    syms = set()
    for o in objs:
        r = subprocess.run(["nm", "-u", o], capture_output=True, text=True, check=True)
        syms.update(re.findall(r"\b(__hip_fatbin_[0-9a-f]+)\b", r.stdout))
    blobs = os.path.join(OUT_DIR, "fatbin_blobs.cpp")
    with open(blobs, "w") as f:
        f.write("// empty device-code blobs of the host-only objects (generated)\n")
        for s in sorted(syms):
            f.write(f'extern "C" const char {s}[16] = {{0}};\n')
    objs.append(_compile_plain(blobs))
    tmp = LIB + ".tmp"
    r = subprocess.run([CLANG, "-shared", "-fsanitize=address,undefined", "-shared-libasan", "-o", tmp] + objs,
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


def _compile_plain(src: str) -> str:
    obj = src + ".o"
    r = subprocess.run([CLANG, "-c", "-fPIC", src, "-o", obj], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{r.stderr}")
    return obj


if __name__ == "__main__":
    print(build())
