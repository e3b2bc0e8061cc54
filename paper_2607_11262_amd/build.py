"""Build libgts.so in-tree with hipcc for gfx950.

    python -m paper_2607_11262_amd.build

Compiles every source each time it is called (the build check must see
compile errors even when a library is already present)."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libgts.so")
BUILD = os.path.join(ROOT, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = os.environ.get("GTS_OFFLOAD_ARCH", "gfx950")

# Packed FP32 instructions are kept out of generated code (-packed-fp32-ops).
DEVICE_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang",
                "-packed-fp32-ops", "-Wall", "-Wno-unused-function"]
# (source, extra flags, object): the windowed kernel's three modes compile
# as parts of their own, side by side
KERNELS = (("gts_sim.hip", (), "gts_sim.o"),
           ("gts_window.hip", ("-DGTS_WINDOW_PART=0",), "gts_window0.o"),
           ("gts_window.hip", ("-DGTS_WINDOW_PART=1",), "gts_window1.o"),
           ("gts_window.hip", ("-DGTS_WINDOW_PART=2",), "gts_window2.o"),
           ("gts_noalloc.hip", (), "gts_noalloc.o"))
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]


def _run(cmd):
    print("+", " ".join(cmd), flush=True)
    subprocess.check_call(cmd)


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    objs = []
    for src, extra, obj in KERNELS:
        o = os.path.join(BUILD, obj)
        jobs.append([HIPCC, *DEVICE_FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", o])
        objs.append(o)
    host_o = os.path.join(BUILD, "gts_host.o")
    jobs.append([HIPCC, *HOST_FLAGS, "-x", "c++", "-c", os.path.join(CSRC, "gts_host.cpp"), "-o", host_o])
    # the sources compile independently: all at once
    procs = []
    for cmd in jobs:
        print("+", " ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd)))
    failed = [cmd for cmd, p in procs if p.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, failed[0])
    tmp = OUT + f".tmp{os.getpid()}"
    _run([HIPCC, "-shared", f"--offload-arch={ARCH}", "-fPIC", "-o", tmp, *objs, host_o])
    os.replace(tmp, OUT)
    return OUT


def build_host_sanitized(out: str) -> str:
    """A CPU-only build of the host library (validation, device image
    construction, argument checks) with g++ under AddressSanitizer and
    UBSan, kernel launches replaced by stand-ins that report no device.
    Load it into a process started with the sanitizer runtimes preloaded."""
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__",
           "-I/opt/rocm/include", os.path.join(CSRC, "gts_host.cpp"), os.path.join(CSRC, "gts_host_only.cpp"),
           "-L/opt/rocm/lib", "-lamdhip64", "-o", out]
    _run(cmd)
    return out


if __name__ == "__main__":
    build()
    sys.exit(0)
