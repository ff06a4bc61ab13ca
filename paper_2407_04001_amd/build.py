"""Build libpase.so (host planner + gfx950 kernels) in-tree with hipcc.

The sources are compiled to objects in parallel, then linked."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libpase.so")
ARCH = "gfx950"

# Every HIP compile disables packed FP32 instruction selection (no v_pk_*_f32).
HIP_FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-fno-honor-nans", "-Wall", "-Wno-unused-function"]


def sources():
    return [os.path.join(CSRC, f) for f in ("host.cpp", "launch_plan.cpp", "assign.cpp", "device.hip")]


def build(verbose: bool = False, out: str = LIB, extra=()) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    objs, procs = [], []
    for src in sources():
        obj = out + "." + os.path.splitext(os.path.basename(src))[0] + ".o"
        cmd = [hipcc, *HIP_FLAGS, *inc, "-c", src, "-o", obj, *extra]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((subprocess.Popen(cmd), cmd))
        objs.append(obj)
    failed = [cmd for p, cmd in procs if p.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, failed[0])
    tmp = out + ".tmp"
    cmd = [hipcc, *HIP_FLAGS, "-shared", *objs, "-o", tmp, *extra]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    for obj in objs:
        os.remove(obj)
    return out


# Host-only build of the planner (host.cpp, launch_plan.cpp, assign.cpp) with a stub
# device runtime, under AddressSanitizer and UBSan, for the CPU test suite.
# The GPU library is never built this way: this is g++ on host sources only.
SAN_LIB = os.path.join(ROOT, "_build", "libpase_host_san.so")
SAN_FLAGS = ["-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wall", "-Wno-unused-function"]


def build_host_sanitized(out: str = SAN_LIB, verbose: bool = False) -> str:
    os.makedirs(os.path.dirname(out), exist_ok=True)
    srcs = [os.path.join(CSRC, f) for f in ("host.cpp", "launch_plan.cpp", "assign.cpp", "device_stub.cpp")]
    cmd = [os.environ.get("CXX", "g++"), *SAN_FLAGS, "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           *srcs, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
