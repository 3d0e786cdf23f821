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


DEVICE_SOURCES = ("kamera_kernels.hip", "kamera_rows.hip", "kamera_patch.hip")


def build(verbose: bool = False, save_temps: bool = False) -> str:
    """Compile the kernels and the host ABI layer (the objects in parallel) and
    link libkamera.so."""
    from concurrent.futures import ThreadPoolExecutor

    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    common = ["-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC]
    cmds, objs = [], []
    for src in DEVICE_SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc, "-c", "-O3", f"--offload-arch={ARCH}", *NO_PACKED_FP32, *common,
               "-Wno-unused-command-line-argument", os.path.join(CSRC, src), "-o", obj]
        if save_temps:
            cmd.insert(2, "-save-temps=obj")
        cmds.append(cmd)
        objs.append(obj)
    # the ABI layer is plain host C++: validation and launch set-up only
    aobj = os.path.join(BUILD, "kamera_abi.o")
    cmds.append(["g++", "-c", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                 *common, os.path.join(CSRC, "kamera_abi.cpp"), "-o", aobj])
    objs.append(aobj)
    with ThreadPoolExecutor(max_workers=len(cmds)) as ex:
        for f in [ex.submit(_run, c, verbose) for c in cmds]:
            f.result()
    tmp = LIB + ".tmp"
    _run([hipcc, "-shared", f"--offload-arch={ARCH}", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    build_ceiling(verbose)
    return LIB


CEILING_LIB = os.path.join(PKG, "libkamera_ceiling.so")


def build_ceiling(verbose: bool = False) -> str:
    """libkamera_ceiling.so: the benchmark's same-traffic copy kernel (a
    measurement of the device, not part of the operator's library)."""
    hipcc = _hipcc()
    tmp = CEILING_LIB + ".tmp"
    _run([hipcc, "-shared", "-O3", f"--offload-arch={ARCH}", *NO_PACKED_FP32, "-std=c++17", "-fPIC",
          "-Wno-unused-command-line-argument", os.path.join(CSRC, "kamera_ceiling.hip"), "-o", tmp], verbose)
    os.replace(tmp, CEILING_LIB)
    return CEILING_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, save_temps="--save-temps" in sys.argv))
