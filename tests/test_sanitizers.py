"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Three programs are built with gcc/g++ and the sanitizers and run to completion:
  - tests/sanitize_driver.c: every entry point of the fp64 oracle on small
    random batches whose buffers are allocated to their exact sizes;
  - tests/plan_check.cpp: the host planner's work split and its replay of
    every worker walk and merge lookup;
  - tests/table_check_driver.cpp: the debug build's block-id check.
Any out-of-bounds access, leak or undefined operation aborts the program
(-fno-sanitize-recover), which fails the test.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _env():
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "sanitize_driver")
    subprocess.run(["gcc", *SAN, "-std=c11", "-o", exe, os.path.join(HERE, "sanitize_driver.c"), "-lm"],
                   check=True)
    r = subprocess.run([exe, "60"], capture_output=True, text=True, timeout=300, env=_env())
    assert r.returncode == 0, r.stderr[-4000:]
    assert r.stdout.startswith("OK"), r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not found")
def test_planner_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "plan_check")
    subprocess.run(["g++", *SAN, "-std=c++17", "-o", exe, os.path.join(HERE, "plan_check.cpp")], check=True)
    r = subprocess.run([exe, "150", "3"], capture_output=True, text=True, timeout=600, env=_env())
    assert r.returncode == 0, r.stderr[-4000:]
    assert r.stdout.startswith("OK"), r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not found")
def test_block_id_check_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "table_check")
    subprocess.run(["g++", *SAN, "-std=c++17", "-o", exe, os.path.join(HERE, "table_check_driver.cpp")], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=_env())
    assert r.returncode == 0, r.stdout + r.stderr[-4000:]
    assert "all table checks passed" in r.stdout
