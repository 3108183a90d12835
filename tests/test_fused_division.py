"""The fused on-the-fly mode quantizes with a reciprocal and one residual step instead of a
division.  This CPU test runs tests/c/recip_division_check.c, which compares that quotient with
the correctly rounded FP32 division for every FP16 input pair the quantization rule can meet
(about 1e9 pairs, a few seconds), and checks that the clamp to [-127, 127] never acts."""

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_reciprocal_residual_division_is_exact(tmp_path):
    exe = tmp_path / "recip_division_check"
    # -ffp-contract=off: only the fmaf calls fuse; -O2 keeps the sweep to seconds
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-o", str(exe),
                    os.path.join(HERE, "c", "recip_division_check.c"), "-lm"], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stdout + out.stderr
    assert "mismatches 0 out_of_range 0" in out.stdout
    pairs = int(out.stdout.split()[1])
    assert pairs > 10 ** 9
