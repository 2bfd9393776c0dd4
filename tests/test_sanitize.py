"""The scheduler (schedule.cpp) and the oracle's C loops (oracle.c) built
for the host with AddressSanitizer and UndefinedBehaviorSanitizer, driven
over a grid of descriptors and their plans (tests/sanitize/plan_grid.cpp).
Host code only: nothing here is built for or run on a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None,
                    reason="needs gcc and g++")
def test_scheduler_and_oracle_under_sanitizers(tmp_path):
    obj = str(tmp_path / "oracle.o")
    exe = str(tmp_path / "plan_grid")
    subprocess.check_call(["gcc", "-std=c11", "-c", *SAN, "-o", obj,
                           os.path.join(ROOT, "oracle", "oracle.c")])
    subprocess.check_call(["g++", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "include"),
                           "-o", exe, os.path.join(ROOT, "tests", "sanitize", "plan_grid.cpp"),
                           os.path.join(ROOT, "paper_2204_03418_amd", "csrc", "schedule.cpp"),
                           obj, "-lm", "-lgomp"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "0 failed checks" in r.stdout
