"""Build step of the HIP library: one hipcc invocation for gfx950."""
from __future__ import annotations

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libmoe_budget.so")
SOURCES = ["kernels.hip", "prefill.hip", "attention.hip", "residency.cpp", "residency_dev.hip", "capi.cpp", "stack.cpp",
           "analysis.cpp"]
# Host-only sources (the host tier's CPU GEMVs): built by the host compiler, then linked into the library.
HOST_SOURCES = ["host_ffn.cpp"]
HOST_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall", "-Wextra", "-pthread"]
BUILD_DIR = os.path.join(PKG, "_build")

# Packed fp32 ops stay off: the compiler would otherwise form v_pk_* fp32 ops
# from scalar float code.  Hidden visibility exports only the MOE_API entry points.
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-fvisibility=hidden",
               "-Wall", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the library)")


def host_cxx() -> str:
    for cand in (os.environ.get("CXX"), shutil.which("g++"), shutil.which("c++")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("no host C++ compiler found")


def build(verbose: bool = False) -> str:
    """Compile libmoe_budget.so in the package directory; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
        res = subprocess.run([host_cxx(), *HOST_FLAGS, "-I", os.path.join(ROOT, "include"), "-c", "-o", obj,
                              os.path.join(CSRC, src)], capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"host compile of {src} failed ({res.returncode}):\n{res.stderr[-8000:]}")
        objs.append(obj)
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), "-o", tmp,
           *[os.path.join(CSRC, s) for s in SOURCES], "-x", "none", *objs, "-pthread",
           "-Wl,--version-script=" + os.path.join(CSRC, "exports.map")]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stderr[-8000:]}")
    if verbose and res.stderr:
        print(res.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
