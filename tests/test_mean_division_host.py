"""The lookup divides a mean bag's sums by one correctly rounded reciprocal of
the bag length and one fma correction per element, claiming the IEEE binary32
quotient.  This CPU test builds a small C program (gcc, libm fmaf) that runs
the same three steps and compares them bit for bit with float division over
every sampled significand of several binades, random pairs and exact
quotients.  The GPU-side counterpart is tests/test_gpu_mean_division.py."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_reciprocal_correction_equals_ieee_division(tmp_path):
    exe = tmp_path / "mean_division_check"
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-o", str(exe),
                    os.path.join(HERE, "host", "mean_division_check.c"), "-lm"], check=True)
    r = subprocess.run([str(exe), "2000000", "7"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "mismatches 0" in r.stdout
