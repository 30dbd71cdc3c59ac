"""The library's host code (plan validation and tables, the P:D planner, the
pipe's argument checks) built with g++ under AddressSanitizer and
UndefinedBehaviorSanitizer and driven by tests/host_fuzz.cpp: random and
mostly-valid descriptors (every head map, order, dtype, cache type and layer
range), block-table checks, segment queries and planner problems.  Runs on
the CPU: without a device every plan is host-only."""
import os
import shutil
import subprocess

import pytest

from conftest import ROOT

CSRC = os.path.join(ROOT, "paper_2509_17542_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists("/opt/rocm/lib"),
                    reason="needs g++ and the ROCm runtime library")
def test_host_code_under_sanitizers(tmp_path):
    exe = tmp_path / "host_fuzz"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "host_fuzz.cpp"), os.path.join(CSRC, "kvx_plan.cpp"),
           os.path.join(CSRC, "kvx_pd.cpp"), os.path.join(CSRC, "kvx_pipe.cpp"),
           "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "Sanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
    assert "plans ok" in r.stdout
