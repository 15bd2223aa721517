"""Division by the block-decoding run's divisors as a multiplication
(paper_2007_13005_amd/csrc/smol_magic.h, used to map the kernel's job indices
to blocks) against integer division on the CPU: every divisor up to 2^16 at
and around its multiples and at the ends of the numerator range (< 2^31), and
seeded large divisors (tests/csrc/magic_check.cpp)."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_magic_division_matches_integer_division(tmp_path):
    exe = tmp_path / "magic_check"
    cmd = ["g++", "-std=c++17", "-O2", "-I", os.path.join(ROOT, "paper_2007_13005_amd", "csrc"),
           os.path.join(ROOT, "tests", "csrc", "magic_check.cpp"), "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stderr[-4000:]
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stdout[-2000:]
    assert res.stdout.startswith("checks "), res.stdout
