"""The host layer (csrc/glance_api.cpp: argument checks, plans, workspace
carve-up) built for the CPU with AddressSanitizer and UndefinedBehaviorSanitizer,
its kernel launchers replaced by host stubs that check the carve-up against
the kernels' largest indices (tests/host_sanitize/), and driven through every
entry point with accepted and rejected arguments.  No GPU and no HIP runtime
are involved."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "host_sanitize")
ROCM_INCLUDE = "/opt/rocm/include"


def test_host_layer_under_asan_and_ubsan(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.isdir(os.path.join(ROCM_INCLUDE, "hip")):
        pytest.skip("needs g++ and the HIP headers")
    exe = str(tmp_path / "host_driver")
    cmd = [gxx, "-std=c++17", "-g", "-O1", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__",
           "-I", ROCM_INCLUDE, "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2609_00355_amd", "csrc"), "-I", HERE,
           os.path.join(ROOT, "paper_2609_00355_amd", "csrc", "glance_api.cpp"),
           os.path.join(HERE, "stubs.cpp"), os.path.join(HERE, "driver.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "checks passed" in r.stdout
