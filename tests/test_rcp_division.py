"""The row quantizer divides by the group scale through a correctly rounded
reciprocal and one FMA correction; a host program checks, over every bf16
amax the fast path takes and every |x| <= amax, that this gives the divide's
quotient wherever an E4M3 code depends on it (host only, no GPU)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_reciprocal_quotient_equals_divide(tmp_path):
    exe = str(tmp_path / "rcp_division_check")
    subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-o", exe,
                    os.path.join(HERE, "rcp_division_check.c"), "-lm"], check=True)
    out = subprocess.run([exe], capture_output=True, text=True, timeout=600)
    assert out.returncode == 0, out.stdout + out.stderr
    assert "mismatches 0" in out.stdout
