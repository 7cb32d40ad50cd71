"""The library's host code (allocator, planner, status) under AddressSanitizer
and UndefinedBehaviorSanitizer, CPU only.

Builds ``tests/native/host_check.cpp`` against the host sources with g++ and
runs it: random alloc/free/mark_used streams on every policy with the ABI's
invariants checked after every call, random single and batch plans checked
for reassembly and maximality, and every bad-argument path.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2504_03775_amd", "csrc")
HOST_SOURCES = ["flowkv_status.cpp", "flowkv_alloc.cpp", "flowkv_plan.cpp", "flowkv_sched.cpp"]


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_code_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "host_check")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "native", "host_check.cpp"),
           *[os.path.join(CSRC, s) for s in HOST_SOURCES], "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, timeout=300)
    # verify_asan_link_order=0: the sanitizer runtime need not be the first
    # library loaded, so the process environment is passed on unchanged
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, "150"], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "rounds ok" in r.stdout
