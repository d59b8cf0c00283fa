"""The planner and the controller (host C++, no HIP calls) under the address
and undefined-behaviour sanitizers: tests/native/host_fuzz.cpp is built with
g++ against plan.cpp and controller.cpp and run on random valid and invalid
inputs. Skipped when g++ or its sanitizer runtimes are missing."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_04415_amd", "csrc")


def test_planner_and_controller_under_sanitizers():
    gxx = shutil.which("g++")
    if not gxx:
        pytest.skip("g++ not found")
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "host_fuzz")
        cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
               "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
               os.path.join(ROOT, "tests", "native", "host_fuzz.cpp"), os.path.join(CSRC, "plan.cpp"),
               os.path.join(CSRC, "controller.cpp"), "-o", exe]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0 and "sanitizer" in (r.stderr or "").lower():
            pytest.skip("sanitizer runtime unavailable: " + r.stderr[-300:])
        assert r.returncode == 0, r.stderr[-3000:]
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
                   UBSAN_OPTIONS="print_stacktrace=1")
        r = subprocess.run([exe, "3000"], capture_output=True, text=True, env=env, timeout=300)
        assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
        assert "plans ok" in r.stdout
