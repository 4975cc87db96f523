"""The host planner (csrc/rnnt_arc_plan.cpp, which turns caller-supplied arc
lists into the device image's offset tables) built on its own with the address
and undefined-behaviour sanitizers, and every case of test_arc_plan_cpu.py --
the replays against the oracle, the rejected lists and the seeded fuzz of random
and malformed arc lists -- run against that build in a child process that
preloads the sanitizer runtime.  CPU only: the build uses g++ and no device code.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2303_10384_amd", "csrc", "rnnt_arc_plan.cpp")


def test_planner_cases_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    so = str(tmp_path / "librnnt_arc_plan_sanitized.so")
    # host C++ only; the HIP runtime header is read for its types, no device code is built
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wall",
           "-D_GLIBCXX_ASSERTIONS",  # bounds-checked std::vector indexing as well
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__",
           SRC, "-o", so]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    runtime = subprocess.run([gxx, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    assert os.path.isabs(runtime) and os.path.exists(runtime), runtime
    env = dict(os.environ)
    env.update(LD_PRELOAD=runtime, RNNT_ARC_PLAN_SANITIZED=so,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # -s: no output capture in the child, so a sanitizer report reaches this test's message
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-s", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_arc_plan_cpu.py")],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-6000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert " passed" in res.stdout and "skipped" not in res.stdout.split("\n")[-2], res.stdout[-2000:]
