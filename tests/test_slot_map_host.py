"""The attention kernel's launch-slot map (slot_map.h) on the host, built
with g++ under AddressSanitizer and UndefinedBehaviorSanitizer: for equal
and work-balanced XCD-group shares over thousands of task counts, run
lengths and work distributions, every task has exactly one slot and the
balanced shares of equal-work heads are equal in count."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2609_25869_amd", "csrc")


def test_every_task_has_exactly_one_slot(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "slot_map_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", CSRC, os.path.join(HERE, "sanitize", "slot_map_driver.cpp"), "-o", exe]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
    assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout[-2000:]
