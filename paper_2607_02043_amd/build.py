"""Build libmlastep.so (gfx950 HIP kernels + C ABI) in place, next to this file."""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmlastep.so")
SOURCES = ["mla_kernels.hip", "mla_api.cpp", "proj_kernels.hip", "proj_api.cpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", INCLUDE, "-I", CSRC,
]


TRACE_LIB = os.path.join(PKG, "libmlastep_trace.so")


def build(verbose: bool = False, trace: bool = False) -> str:
    """Compile the library; trace=True builds the profiling variant
    (libmlastep_trace.so: the attention kernel also records a per-item
    timeline, read by timeline.py) instead."""
    objs = []
    lib = TRACE_LIB if trace else LIB
    for src in SOURCES:
        obj = os.path.join(CSRC, src + (".trace.o" if trace else ".o"))
        cmd = [HIPCC, *FLAGS, *(["-DMLA_TRACE"] if trace else []), "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    tmp = lib + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    for o in objs:
        os.remove(o)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, trace="--trace" in sys.argv))
