"""The host C++ of the path (the attention planner and the scheduler) built
with AddressSanitizer and UndefinedBehaviorSanitizer and driven over random
inputs on the CPU: any out-of-bounds access, use after free, leak or
undefined operation aborts the driver."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_09061_amd", "csrc")
FLAGS = ["-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")


def _build_and_run(tmp_path, driver, sources):
    exe = str(tmp_path / driver.replace(".cpp", ""))
    cmd = ["g++", *FLAGS, os.path.join(ROOT, "tests", "native", driver),
           *[os.path.join(CSRC, s) for s in sources], "-o", exe]
    subprocess.run(cmd, check=True, timeout=300)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    return r.stdout


def test_planner_under_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, "plan_fuzz.cpp", ["plan.cpp"])
    assert out.startswith("ok")


def test_scheduler_under_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, "sched_fuzz.cpp", ["sched.cpp"])
    assert out.count("pending 0") == 8
