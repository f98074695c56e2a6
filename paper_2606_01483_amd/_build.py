"""Build libmurmur.so for gfx950 (MI355X) from csrc/.

kernels.hip is compiled by hipcc for gfx950 only; api.cpp (host-only C ABI
layer) by g++.  The shared object lands next to this file, where the ctypes
binding loads it.  Packed-fp32 instruction selection is disabled for device
code, and the first 16 kernel-argument dwords are preloaded into SGPRs.  Only
the murmur_* entry points are exported.
"""
from __future__ import annotations

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmurmur.so")
BUILD_DIR = os.path.join(ROOT, "_build")
ARCH = "gfx950"


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP toolchain (ROCm) is required to build libmurmur")


def _run(cmd: list[str]) -> None:
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"build step failed ({res.returncode}): {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")


COMMON_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", f"-I{INCLUDE}", f"-I{CSRC}", "-Wall"]
# Device code: packed-fp32 instruction selection off; the first 16 kernel-argument dwords preloaded into SGPRs.
KERNEL_FLAGS = [f"--offload-arch={ARCH}", *COMMON_FLAGS, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-kernarg-preload-count=16"]


def build(verbose: bool = False) -> str:
    """Compile every source and link libmurmur.so (always rebuilds)."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    hipcc = _hipcc()
    k_obj = os.path.join(BUILD_DIR, "kernels.o")
    a_obj = os.path.join(BUILD_DIR, "api.o")
    steps = [
        [hipcc, *KERNEL_FLAGS, "-c", os.path.join(CSRC, "kernels.hip"), "-o", k_obj],
        ["g++", *COMMON_FLAGS, "-Wextra", "-c", os.path.join(CSRC, "api.cpp"), "-o", a_obj],
    ]
    for cmd in steps:
        if verbose:
            print(" ".join(cmd), flush=True)
        _run(cmd)
    tmp = LIB + ".tmp"
    link = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", k_obj, a_obj, "-o", tmp]
    if verbose:
        print(" ".join(link), flush=True)
    _run(link)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
