"""The library's host code under the address and undefined-behaviour
sanitizers, on the CPU: validation, geometry and planning (smol_host.cpp),
Algorithm 1's rectangle and the JPEG calls' host side (smol_jpeg.cpp) and the
T.81 stream parser and entropy decoder (smol_jpeg_entropy.cpp) are built with
g++ and -fsanitize=address,undefined against a host-only stand-in for the HIP
runtime (tests/csrc/hip_stub, tests/csrc/host_stub.cpp: no device, so every
call that passes validation ends before it would launch). The driver
(tests/csrc/host_fuzz.cpp) decodes seed JPEG streams -- seeded photo-like
images at several sizes, qualities and restart intervals, encoded by libjpeg
through PIL, plus hand-cut edge streams -- and seeded byte mutations of each
(substitutions, bit flips, spurious 0xFF and restart markers, insertions,
deletions, truncations), whole, through a rectangle and into the rectangle's
MCU window, then makes seeded random calls of the C ABI's validation and
geometry. A sanitizer report stops the run at the first fault."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

from paper_2007_13005_amd import synthetic

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2007_13005_amd", "csrc")
HOST_SOURCES = ["smol_host.cpp", "smol_jpeg.cpp", "smol_jpeg_entropy.cpp"]


def _seed_streams() -> list[bytes]:
    streams = []
    for sizes, seed, quality, restart in [
            ([(48, 32), (64, 64), (127, 93)], 5, 75, 0),
            ([(320, 240), (17, 300), (300, 17)], 6, [50, 90, 100], 1),
            ([(96, 80), (33, 47)], 7, 30, 3),
            ([(1, 1), (16, 16), (200, 8)], 8, 95, 2)]:
        streams += synthetic.jpeg_files(sizes, seed, quality, restart_blocks=restart)
    s = streams[3]
    streams += [s[:len(s) // 2], s[:-2], s[2:], s[:20], b"\xff\xd8\xff\xd9", b""]
    return streams


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "host_fuzz"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "tests", "csrc", "hip_stub"),
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           *[os.path.join(CSRC, f) for f in HOST_SOURCES],
           os.path.join(ROOT, "tests", "csrc", "host_stub.cpp"),
           os.path.join(ROOT, "tests", "csrc", "host_fuzz.cpp"),
           "-o", str(exe), "-lpthread"]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    files = []
    for i, s in enumerate(_seed_streams()):
        p = tmp_path / f"seed{i:02d}.jpg"
        p.write_bytes(s)
        files.append(str(p))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([str(exe), "13005", "300", "20000", *files], capture_output=True,
                         text=True, timeout=600, env=env)
    report = res.stderr[-6000:]
    assert res.returncode == 0, report
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, report
    assert res.stdout.startswith("streams "), res.stdout
    # the seeds themselves decode (the mutations mostly do not)
    assert int(res.stdout.split()[3]) >= 16, res.stdout
