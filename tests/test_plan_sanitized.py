"""The planner (csrc/plan.cpp, no HIP) built for the host with
AddressSanitizer and UndefinedBehaviorSanitizer and driven by a seeded fuzz
of graphs and mutation records (tests/native/plan_fuzz.cpp): no memory error,
no undefined behaviour, and the invariants of Algorithm 1 on every accepted
plan."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_planner_under_asan_ubsan(tmp_path):
    exe = tmp_path / "plan_fuzz"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I" + os.path.join(ROOT, "paper_2607_18582_amd", "csrc"),
           os.path.join(ROOT, "tests", "native", "plan_fuzz.cpp"),
           os.path.join(ROOT, "paper_2607_18582_amd", "csrc", "plan.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe), "3000"], capture_output=True, text=True, timeout=300, env=env)
    print(r.stdout[-500:])
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-3000:])
    assert "failures 0" in r.stdout and "ERROR" not in r.stderr
    accepted = int(r.stdout.split("plans accepted ")[1].split(",")[0])
    assert accepted > 1000
