"""The encoders take the tensor scale fl32(amax / 2688) (Section 2, NVFP4 global
scale) as one multiplication by the binary32 reciprocal and one fused correction
by the exact remainder instead of an IEEE division.  This host test compiles a
small C check and confirms the identity against correctly rounded division on a
dense sample of binary32 amax values from 2^-100 up (every binade, four whole
binades); the full range was also checked once, exhaustively."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_two_fma_division_by_2688(tmp_path):
    exe = str(tmp_path / "sg_division")
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-o", exe,
                    os.path.join(HERE, "native", "sg_division.c"), "-lm"], check=True)
    out = subprocess.run([exe, "61"], check=True, capture_output=True, text=True).stdout.split()
    bad, n = int(out[0]), int(out[1])
    assert n > 60_000_000
    assert bad == 0
