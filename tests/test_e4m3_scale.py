"""The encoders round block scales to E4M3 from the bit pattern of the quotient
(Section 2, NVFP4 block scale; E4M3 round to nearest even) and take the quotient as
bmax * rcp(den) away from E4M3 midpoints.  This host test compiles a small C check:
the bit rounding against the nearest point of the E4M3 grid for every binary32 in
[0, 448], and the quotient shortcut against the correctly rounded quotient for
random and midpoint-seeking operands with reciprocals up to one ulp off."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_e4m3_rounding_and_quotient_shortcut(tmp_path):
    exe = str(tmp_path / "e4m3_scale")
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-o", exe,
                    os.path.join(HERE, "native", "e4m3_scale.c"), "-lm"], check=True)
    bad1, bad2, tried = (int(v) for v in subprocess.run([exe], check=True, capture_output=True,
                                                         text=True).stdout.split())
    assert bad1 == 0
    assert tried > 5_000_000
    assert bad2 == 0
