"""The C ABI layer built for the host alone, under AddressSanitizer and
UndefinedBehaviorSanitizer, with the kernels and the HIP runtime replaced by recording stubs
(tests/host/nq_abi_host.cpp): argument validation, error propagation (a failing launch or
device query is NQ_ERR_HIP), dispatch to the launcher each call's contract names, and
per-thread error messages.  CPU only."""

import os
import shutil
import subprocess

import pytest

from conftest import ROOT

CSRC = os.path.join(ROOT, "paper_2502_09720_amd", "csrc")


def test_abi_layer_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.isdir("/opt/rocm/include"):
        pytest.skip("needs g++ and the ROCm headers")
    exe = str(tmp_path / "nq_abi_host")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-Wall",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
           "-I", CSRC, os.path.join(ROOT, "tests", "host", "nq_abi_host.cpp"),
           os.path.join(CSRC, "nq_api.cpp"), os.path.join(CSRC, "nq_host.cpp"), "-o", exe,
           "-lpthread"]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    # verify_asan_link_order=0: another preloaded library may come before the ASan runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "all host ABI checks passed" in run.stdout
