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


CLANG = os.environ.get("LOGBQ_HOST_CLANG", "/opt/rocm/llvm/bin/clang++")


def build_sanitized(sanitize: str, verbose: bool = False) -> str:
    """A CPU-test build of liblogbq.so with LLVM sanitizers on its host code: `sanitize` is
    "address,undefined" or "thread". The host fit (fit.cpp) and the host side of the kernel
    source (argument checks, tables, launches) are instrumented; device code is not. The
    library lands in _build/san_<kinds>/ and needs the matching runtime preloaded, e.g.
    LD_PRELOAD=$(clang++ -print-file-name=libclang_rt.asan-x86_64.so) for address; point the
    binding at it with LOGBQ_LIBRARY=<path>."""
    tag = sanitize.replace(",", "_")
    out_dir = os.path.join(BUILD, f"san_{tag}")
    os.makedirs(out_dir, exist_ok=True)
    san = [f"-fsanitize={sanitize}", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-g", "-shared-libsan"]
    fit_o = os.path.join(out_dir, "fit.o")
    ker_o = os.path.join(out_dir, "logbq_kernels.o")
    host_flags = [f for f in HOST_FLAGS if f != "-O2"] + ["-O1"]
    _run([CLANG, *host_flags, *san, "-c", os.path.join(CSRC, "fit.cpp"), "-o", fit_o], verbose)
    _run([HIPCC, *HIP_FLAGS, *[a for f in san for a in ("-Xarch_host", f)], "-c",
          os.path.join(CSRC, "logbq_kernels.hip"), "-o", ker_o], verbose)
    lib = os.path.join(out_dir, "liblogbq.so")
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *san, "-o", lib, fit_o, ker_o],
         verbose)
    return lib


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        print(build_sanitized(sys.argv[sys.argv.index("--sanitize") + 1], verbose="-v" in sys.argv))
    else:
        print(build(verbose="-v" in sys.argv))
