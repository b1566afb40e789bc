"""The host planner under AddressSanitizer and UndefinedBehaviorSanitizer.

``tests/planner_sanitizer_driver.cpp`` builds plans (tile lists, XCD splits,
workspace layout, stable-rank tables) for the benchmark sets, for edge-case
lists and for 60 seeded random lists, and checks each plan's work lists: every
XCD split partitions its list, the symmetric products hold each lower-triangle
tile once, and the apply's two lists cover each padded output exactly once.
This test compiles it with ``plan.cpp`` by g++ with both sanitizers and fails on
any sanitizer report, rejected plan or violated invariant. Host code only: no
HIP call.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2605_19811_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_planner_clean_under_host_sanitizers(tmp_path):
    exe = str(tmp_path / "planner_sanitized")
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{CSRC}",
           os.path.join(HERE, "planner_sanitizer_driver.cpp"), os.path.join(CSRC, "plan.cpp"),
           "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0 and "asan" in (res.stderr + res.stdout).lower():
        pytest.skip("sanitizer runtime not available: " + res.stderr[-300:])
    assert res.returncode == 0, res.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    out = run.stdout + run.stderr
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-3000:]
    assert run.returncode == 0, out[-3000:]
    assert "failures 0" in run.stdout
