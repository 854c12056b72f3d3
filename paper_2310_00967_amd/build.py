"""Builds the gfx950 sparsify library in-tree: paper_2310_00967_amd/libmicro_sparsify.so.

hipcc compiles the kernel (device + host stub) and the host library
separately, then links one shared object whose exported symbols are exactly
the C ABI of include/micro_sparsify.h.  Floating point: no contraction
(-ffp-contract=off), no fast-math, subnormals kept, correctly rounded binary32
division, and the packed-fp32 instructions disabled for device code.
"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libmicro_sparsify.so")
ARCH = "gfx950"


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


COMMON = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-fast-math",
          "-Wall", "-Wextra", f"-I{INCLUDE}", f"-I{CSRC}"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-fhip-fp32-correctly-rounded-divide-sqrt", "-fvisibility=hidden"]
KERNEL_SOURCES = ["sparsify_kernel.hip", "union_kernel.hip", "static_scratch.hip", "topk_kernel.hip"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build_library(verbose=False, extra_device_flags=()):
    """Compiles every HIP source for gfx950 (every call) and returns the .so path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    cc = hipcc()
    kobjs = []
    for src in KERNEL_SOURCES:
        obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
        _run([cc, *COMMON, *DEVICE, *extra_device_flags, "-x", "hip", "-c",
              os.path.join(CSRC, src), "-o", obj], verbose)
        kobjs.append(obj)
    hobj = os.path.join(BUILD_DIR, "micro_sparsify.o")
    _run([cc, *COMMON, "-fvisibility=hidden", "-c", os.path.join(CSRC, "micro_sparsify.cpp"),
          "-o", hobj], verbose)
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *kobjs, hobj], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True or "-v" in sys.argv))
