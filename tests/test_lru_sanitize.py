"""Build the host code of the library -- the slot table, the static budget planner and the
offline miss bound -- with AddressSanitizer + UndefinedBehaviorSanitizer (g++) and run
randomised invariant checks over it."""
import os
import shutil
import subprocess

import pytest

from conftest import ROOT


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_slot_table_under_sanitizers(tmp_path):
    exe = tmp_path / "lru_fuzz"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", os.path.join(ROOT, "tests", "lru_fuzz.cpp"),
           os.path.join(ROOT, "paper_2607_09686_amd", "csrc", "slot_lru.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_planner_and_bound_under_sanitizers(tmp_path):
    exe = tmp_path / "host_fuzz"
    csrc = os.path.join(ROOT, "paper_2607_09686_amd", "csrc")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", os.path.join(ROOT, "tests", "host_fuzz.cpp"),
           os.path.join(csrc, "planner.cpp"), os.path.join(csrc, "policy.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok")
