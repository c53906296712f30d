"""Build liblogbq.so in-tree: the host fit with g++, the gfx950 kernels with hipcc. Also builds
libhbmread.so, the streaming-read kernel bench.py measures the HBM read ceiling with.

The host fit is compiled without -ffast-math and with -ffp-contract=off so that its float64
arithmetic rounds exactly as written. All HIP code is compiled with packed-fp32 instructions
disabled (-Xclang -target-feature -Xclang -packed-fp32-ops).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "liblogbq.so")
READ_LIB = os.path.join(HERE, "libhbmread.so")
ARCH = os.environ.get("LOGBQ_OFFLOAD_ARCH", "gfx950")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# The GEMV hands out rows with a one-lane LDS atomic whose result it reads only after the next
# row's products; the atomic optimizer would rewrite that atomic into a wavefront-wide one that
# reads its result at once, stalling the wavefront on the LDS round trip.
HIP_FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-I", INCLUDE,
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
             "-mllvm", "-amdgpu-kernarg-preload-count=16",
             "-Wall", "-Wno-unused-function"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-fast-math", "-Wall",
              "-I", INCLUDE]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    fit_o = os.path.join(BUILD, "fit.o")
    ker_o = os.path.join(BUILD, "logbq_kernels.o")
    _run(["g++", *HOST_FLAGS, "-c", os.path.join(CSRC, "fit.cpp"), "-o", fit_o], verbose)
    _run([HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, "logbq_kernels.hip"), "-o", ker_o], verbose)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, fit_o, ker_o], verbose)
    os.replace(tmp, LIB)
    tmp = READ_LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-shared", "-o", tmp, os.path.join(CSRC, "hbm_read.hip")], verbose)
    os.replace(tmp, READ_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
