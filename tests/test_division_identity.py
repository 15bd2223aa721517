"""The kernels normalise with q = q0 + (a - std*q0) * y, q0 = a*y, y = RN(1/std)
(two FMAs) instead of an IEEE division. This pins that the sequence returns the
correctly rounded quotient for the divisors used here, over a sample of every
binade the numerator can occupy. Runs on the CPU (gcc, hardware FMA)."""
from __future__ import annotations

import os
import subprocess

import numpy as np
import pytest

from paper_2007_13005_amd import synthetic

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("div") / "div_identity")
    flags = ["-O2", "-ffp-contract=off"]
    probe = subprocess.run(["gcc", "-mfma", "-x", "c", "-", "-o", os.devnull],
                           input="int main(void){return 0;}", capture_output=True, text=True)
    if probe.returncode == 0:
        flags.append("-mfma")
    subprocess.run(["gcc", *flags, "-o", exe, os.path.join(HERE, "csrc", "div_identity.c"),
                    "-lm"], check=True)
    return exe


def test_fma_corrected_quotient_is_correctly_rounded(checker):
    divisors = [repr(float(v)) for v in synthetic.IMAGENET_STD_255] + ["1.0", "3.0", "0.1",
                                                                      "255.0", "77.77"]
    res = subprocess.run([checker, "61", *divisors], capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip().startswith("0 mismatches"), res.stdout


def test_reciprocal_is_fp32_correctly_rounded():
    # The host forms RN(1/std) with an fp32 division; numpy's float32 division
    # is IEEE, so the two agree.
    s = synthetic.IMAGENET_STD_255
    assert np.all(np.float32(1.0) / s == (1.0 / s.astype(np.float64)).astype(np.float32))
