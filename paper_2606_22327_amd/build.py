"""Build the HIP library ``libsvfsim.so`` for gfx950 with hipcc.

The library holds every kernel of the simulator and the host runtime behind
the C ABI of ``include/svfsim.h``, plus the host-side exact optimum of tiny
burst instances (``include/svfopt.h``).  It is built in-tree so that the same file
is loaded by the tests, the smoke check and the benchmark.
"""

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libsvfsim.so")

ARCH = os.environ.get("SVFSIM_ARCH", "gfx950")
# Packed FP32 instructions are kept out of every code object.  Uniform
# branches are left as scalar branches rather than structured with lane masks
# (the simulation kernels are bound by scalar instruction issue).
GPU_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-mllvm", "-structurizecfg-skip-uniform-regions"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I", INCLUDE, "-I", CSRC]


def _run(cmd):
    subprocess.check_call(cmd)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    kern_o = os.path.join(BUILD, "svf_kernels.o")
    rt_o = os.path.join(BUILD, "svf_runtime.o")
    _run(["hipcc", f"--offload-arch={ARCH}", *COMMON, *GPU_FLAGS, "-c",
          os.path.join(CSRC, "svf_kernels.hip"), "-o", kern_o])
    na_o = os.path.join(BUILD, "svf_noalloc.o")
    _run(["hipcc", f"--offload-arch={ARCH}", *COMMON, *GPU_FLAGS, "-c",
          os.path.join(CSRC, "svf_noalloc.hip"), "-o", na_o])
    opt_o = os.path.join(BUILD, "svf_opt.o")
    _run(["hipcc", *COMMON, "-c", os.path.join(CSRC, "svf_runtime.cpp"), "-o", rt_o])
    _run(["hipcc", *COMMON, "-c", os.path.join(CSRC, "svf_opt.cpp"), "-o", opt_o])
    tmp = LIB + ".tmp"
    _run(["hipcc", f"--offload-arch={ARCH}", "-shared", "-fPIC", kern_o, na_o, rt_o, opt_o, "-pthread",
          "-o", tmp])
    os.replace(tmp, LIB)
    if verbose:
        print(LIB)
    return LIB


# The runtime's host code under the address and undefined-behaviour
# sanitizers (device code is not instrumented: each flag goes to the host
# compilation only), for the ABI test driver of tests/native.
SAN_HOST = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
            "-Xarch_host", "-fno-omit-frame-pointer"]
SAN_EXE = os.path.join(BUILD, "abi_asan")


def build_abi_sanitized(verbose: bool = False) -> str:
    """Link tests/native/abi_asan_main.cpp and a sanitized build of the
    runtime with the kernel objects of ``build()`` into ``_build/abi_asan``."""
    kern_o = os.path.join(BUILD, "svf_kernels.o")
    na_o = os.path.join(BUILD, "svf_noalloc.o")
    if not (os.path.exists(kern_o) and os.path.exists(na_o)):
        build()
    flags = ["-O1", "-g", "-std=c++17", "-fPIC", "-Wall", "-I", INCLUDE, "-I", CSRC]
    rt_o = os.path.join(BUILD, "svf_runtime_san.o")
    drv_o = os.path.join(BUILD, "abi_asan_main.o")
    _run(["hipcc", *flags, *SAN_HOST, "-c", os.path.join(CSRC, "svf_runtime.cpp"), "-o", rt_o])
    _run(["hipcc", *flags, *SAN_HOST, "-c", os.path.join(ROOT, "tests", "native", "abi_asan_main.cpp"),
          "-o", drv_o])
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    tmp = SAN_EXE + ".tmp"
    _run([os.path.join(rocm, "llvm", "bin", "clang++"), "-fsanitize=address,undefined", drv_o, rt_o,
          kern_o, na_o, "-L", os.path.join(rocm, "lib"), "-lamdhip64",
          "-Wl,-rpath," + os.path.join(rocm, "lib"), "-pthread", "-o", tmp])
    os.replace(tmp, SAN_EXE)
    if verbose:
        print(SAN_EXE)
    return SAN_EXE


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
