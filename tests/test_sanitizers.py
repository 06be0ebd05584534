"""AddressSanitizer + UndefinedBehaviorSanitizer builds of the host code that runs on the CPU:
the oracle (oracle/nmm_oracle.c) and the planner (csrc/plan.cpp), each driven over small and
edge-case inputs by a driver under tests/sanitize/.  Built with gcc / g++ only (no device code);
any sanitizer finding aborts the driver, and the test fails."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _build_and_run(tmp_path, cmd, exe):
    r = subprocess.run(cmd + ["-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert " 0 failures" in r.stdout, r.stdout
    return r.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    cmd = ["gcc", "-std=c11", *SAN, "-fopenmp", "-ffp-contract=off", os.path.join(ROOT, "oracle", "nmm_oracle.c"),
           os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"), "-lm"]
    _build_and_run(tmp_path, cmd, tmp_path / "oracle_asan")


def test_planner_under_asan_ubsan(tmp_path):
    cmd = ["g++", "-std=c++17", *SAN, f"-I{os.path.join(ROOT, 'include')}",
           f"-I{os.path.join(ROOT, 'paper_2609_16009_amd', 'csrc')}",
           os.path.join(ROOT, "paper_2609_16009_amd", "csrc", "plan.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "plan_driver.cpp")]
    out = _build_and_run(tmp_path, cmd, tmp_path / "plan_asan")
    assert "plans checked" in out
