"""In-tree build of libkvx.so for gfx950 (hipcc, no JIT cache)."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libkvx.so")

# Packed-FP32 instructions are disabled for every HIP translation unit.
HIP_FLAGS = ["-O3", "--offload-arch=gfx950", "-fPIC", "-std=c++17", "-Wall",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
              "-I/opt/rocm/include"]


def sources():
    hip = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    cpp = sorted(f for f in os.listdir(CSRC) if f.endswith(".cpp"))
    return hip, cpp


def build_library(jobs: int = 8) -> str:
    hip, cpp = sources()
    if not hip and not cpp:
        return ""
    objdir = os.path.join(ROOT, "_build", "kvx")
    os.makedirs(objdir, exist_ok=True)
    inc = ["-I" + os.path.join(ROOT, "include"), "-I" + CSRC]
    procs, objs = [], []
    for f in hip:
        o = os.path.join(objdir, f + ".o")
        objs.append(o)
        procs.append(subprocess.Popen(["hipcc", *HIP_FLAGS, *inc, "-c", os.path.join(CSRC, f),
                                       "-o", o], cwd=ROOT))
    for f in cpp:
        o = os.path.join(objdir, f + ".o")
        objs.append(o)
        procs.append(subprocess.Popen(["g++", *HOST_FLAGS, *inc, "-c", os.path.join(CSRC, f),
                                       "-o", o], cwd=ROOT))
    bad = [p.args for p in procs if p.wait() != 0]
    if bad:
        raise RuntimeError(f"compile failed: {bad}")
    tmp = LIB + ".tmp"
    subprocess.run(["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs,
                    "-lpthread", "-L/opt/rocm/lib", "-lhsa-runtime64"], check=True, cwd=ROOT)
    os.replace(tmp, LIB)
    return LIB
