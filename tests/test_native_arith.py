"""Exhaustive checks of arithmetic identities the gfx950 kernels rely on, run on the host CPU
(IEEE fp32, denormals kept, as the kernels run)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def test_linear_step255_equals_ieee_division(tmp_path):
    """The 8-bit linear norm spacing (R'max - R'min) / 255 is computed in the decode and
    attention kernels as a product corrected once by its residual (two fmas, 3 instructions
    instead of the 12 of the division sequence).  Every finite fp32 input must round exactly
    as the IEEE division does."""
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "step255")
    subprocess.run([cc, "-O2", "-fopenmp", "-ffp-contract=off", "-mfma", "-o", exe,
                    os.path.join(HERE, "native", "step255_exhaustive.c"), "-lm"], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "mismatches 0" in r.stdout
