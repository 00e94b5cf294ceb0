"""The C ABI's host code (validation, ring and anchor bookkeeping, read-set
tables, packed plans, the wavefront driver) built with AddressSanitizer and
UndefinedBehaviorSanitizer and driven through every entry point, with
host-only stand-ins for the kernel launches (tests/host_asan).  The
sanitizers instrument host code only; no GPU is used."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_host_code_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "ff_host_asan"
    san = []
    for flag in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined"):
        san += ["-Xarch_host", flag]
    cmd = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-O1", "-g", *san,
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + os.path.join(ROOT, "include"),
           "-I" + os.path.join(ROOT, "paper_2609_32540_amd", "csrc"),
           os.path.join(ROOT, "paper_2609_32540_amd", "csrc", "ff_cache.cpp"),
           os.path.join(ROOT, "tests", "host_asan", "launch_stubs.cpp"),
           os.path.join(ROOT, "tests", "host_asan", "driver.cpp"),
           "-o", str(exe)]
    build = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert build.returncode == 0, build.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "host ABI checks passed" in run.stdout
