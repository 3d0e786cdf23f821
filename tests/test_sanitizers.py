"""The host layer (kamera_abi.cpp: argument validation and launch set-up)
under the CPU sanitizers.  It is compiled with g++ together with stand-in
launches (tests/c/launch_stub.cpp) instead of the GPU kernels, and driven by
tests/c/abi_sanitize.cpp (randomised argument structs for every entry point,
a refused launch, many threads at once) and by the plain C consumer
tests/c/abi_check.c:

* -fsanitize=address,undefined, with undefined behaviour fatal;
* -fsanitize=thread for the concurrent callers.
"""

from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_23581_amd", "csrc")
TC = os.path.join(ROOT, "tests", "c")
HIP_INCLUDE = "/opt/rocm/include"


def _toolchain():
    if shutil.which("g++") is None or shutil.which("gcc") is None:
        pytest.skip("no g++/gcc")
    if not os.path.exists(os.path.join(HIP_INCLUDE, "hip", "hip_runtime_api.h")):
        pytest.skip("no HIP headers for the launch-parameter structs")


def _flags():
    return ["-O1", "-g", "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__", "-I", HIP_INCLUDE, "-I",
            os.path.join(ROOT, "include"), "-I", CSRC, "-I", TC]


def _build(tmp_path, name, sanitize, main_sources, c_main=None):
    exe = str(tmp_path / name)
    objs = []
    if c_main is not None:
        obj = str(tmp_path / (name + "_main.o"))
        subprocess.run(["gcc", "-std=c11", "-c", *_flags(), *sanitize, c_main, "-o", obj], check=True,
                       capture_output=True, text=True)
        objs.append(obj)
    cmd = ["g++", "-std=c++17", *_flags(), *sanitize, os.path.join(CSRC, "kamera_abi.cpp"),
           os.path.join(TC, "launch_stub.cpp"), *main_sources, *objs, "-o", exe, "-pthread"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    return exe


def _run(exe, env_extra):
    env = dict(os.environ)
    env.update(env_extra)
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0 and res.stdout.strip().endswith("ok"), (res.stdout[-2000:], res.stderr[-4000:])


def test_host_layer_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    _toolchain()
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"]
    exe = _build(tmp_path, "abi_sanitize_asan", san, [os.path.join(TC, "abi_sanitize.cpp")])
    _run(exe, {"ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0", "UBSAN_OPTIONS": "print_stacktrace=1"})


def test_c_consumer_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    _toolchain()
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"]
    exe = _build(tmp_path, "abi_check_asan", san, [], c_main=os.path.join(TC, "abi_check.c"))
    _run(exe, {"ASAN_OPTIONS": "detect_leaks=1"})


def test_host_layer_under_thread_sanitizer(tmp_path):
    _toolchain()
    exe = _build(tmp_path, "abi_sanitize_tsan", ["-fsanitize=thread"], [os.path.join(TC, "abi_sanitize.cpp")])
    _run(exe, {"TSAN_OPTIONS": "halt_on_error=1"})
