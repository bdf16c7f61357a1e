"""The batch-planning calls (Alg. 1 allocation, App. B budget, Eq. 4 cost
model and its data-parallel form, the PTL fit of App. A, the length spread
and its moving average) built from their C++ source with AddressSanitizer
and UndefinedBehaviorSanitizer, and driven by tests/host/planner_sanitize.cpp
over seeded random batches and the edge cases of their contracts.  Host code
only: the compiler is g++, no GPU code is built."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_planner_under_address_and_ub_sanitizers(tmp_path):
    exe = str(tmp_path / "planner_san")
    build = subprocess.run(
        ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-fno-omit-frame-pointer", "-I" + os.path.join(ROOT, "include"),
         os.path.join(ROOT, "paper_2605_30859_amd", "csrc", "planner.cpp"),
         os.path.join(HERE, "host", "planner_sanitize.cpp"), "-o", exe],
        capture_output=True, text=True, timeout=300)
    assert build.returncode == 0, build.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
    assert run.returncode == 0 and run.stdout.strip() == "ok", (run.stdout[-1000:], run.stderr[-3000:])
