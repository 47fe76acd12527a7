"""Host logic: the work split and merge lookup, replayed on the CPU (g++)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


def test_work_split_replay(tmp_path):
    exe = str(tmp_path / "plan_check")
    subprocess.run(["g++", "-O2", "-std=c++17", "-o", exe, os.path.join(HERE, "plan_check.cpp")], check=True)
    for seed in (1, 2):
        r = subprocess.run([exe, "600", str(seed)], capture_output=True, text=True, timeout=300)
        assert r.returncode == 0, r.stderr
        assert r.stdout.startswith("OK")
