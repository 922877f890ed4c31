"""The plan's host-side table builder (plan.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer: a small native harness (tests/native/) builds the
tables of every workload shape and of edge shapes, checks their invariants and
the rejection of invalid configurations.  Host code only; built with g++."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HARNESS = os.path.join(ROOT, "tests", "native", "host_tables_check.cpp")
PLAN = os.path.join(ROOT, "paper_2608_02504_amd", "csrc", "plan.cpp")


def test_host_tables_under_asan_and_ubsan(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.isdir("/opt/rocm/include"):
        pytest.skip("g++ or the ROCm headers are not available")
    exe = str(tmp_path / "host_tables_check")
    flags = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__",
             "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"),
             "-I" + os.path.join(ROOT, "paper_2608_02504_amd", "csrc"),
             "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"]
    res = subprocess.run([gxx, *flags, HARNESS, PLAN, "-o", exe], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    # verify_asan_link_order=0: the environment may preload a library ahead of
    # the sanitizer runtime, which ASan would otherwise refuse to start under
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "host tables: ok" in run.stdout
    assert "runtime error" not in run.stderr and "AddressSanitizer" not in run.stderr
