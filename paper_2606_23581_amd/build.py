"""Build libkamera.so (gfx950 HIP kernels + C ABI) in-tree with hipcc."""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libkamera.so")

ARCH = "gfx950"
# hipcc -O3 forms packed-fp32 instructions from plain float code by itself;
# keep them out of every device compile.
NO_PACKED_FP32 = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: install ROCm or set HIPCC")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"build step failed ({res.returncode}): {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return res


def build(verbose: bool = False, save_temps: bool = False) -> str:
    """Compile the kernels and the host ABI layer and link libkamera.so."""
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    kobj = os.path.join(BUILD, "kamera_kernels.o")
    pobj = os.path.join(BUILD, "kamera_patch.o")
    aobj = os.path.join(BUILD, "kamera_abi.o")
    common = ["-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC]
    kcmd = [hipcc, "-c", "-O3", f"--offload-arch={ARCH}", *NO_PACKED_FP32, *common,
            "-Wno-unused-command-line-argument",
            os.path.join(CSRC, "kamera_kernels.hip"), "-o", kobj]
    if save_temps:
        kcmd.insert(2, f"-save-temps={'obj'}")
    _run(kcmd, verbose)
    pcmd = [hipcc, "-c", "-O3", f"--offload-arch={ARCH}", *NO_PACKED_FP32, *common,
            "-Wno-unused-command-line-argument", os.path.join(CSRC, "kamera_patch.hip"), "-o", pobj]
    if save_temps:
        pcmd.insert(2, "-save-temps=obj")
    _run(pcmd, verbose)
    # the ABI layer is plain host C++: validation and launch set-up only
    _run(["g++", "-c", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
          *common, os.path.join(CSRC, "kamera_abi.cpp"), "-o", aobj], verbose)
    tmp = LIB + ".tmp"
    _run([hipcc, "-shared", f"--offload-arch={ARCH}", "-fPIC", kobj, pobj, aobj, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, save_temps="--save-temps" in sys.argv))
