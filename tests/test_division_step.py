"""The quantizer divides in fp32 without a divide instruction: x = X / s32
with one multiply and two fmas on a correctly rounded reciprocal, and the
quotients by the block scales (and by 6 and 7) with a multiply and one fma
on a two-term reciprocal.  tests/division_step.c proves on the CPU,
exhaustively over the operand mantissas the kernel can see, that both give
the IEEE quotient bit for bit, and that zeros keep their sign."""
import os
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_division_step_exhaustive():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "division_step")
        subprocess.run(["gcc", "-O2", "-mfma", "-std=c11", "-o", exe,
                        os.path.join(HERE, "division_step.c"), "-lm", "-lpthread"], check=True)
        r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "A: 0 of" in r.stdout and "B: 0 of" in r.stdout and "C: 0 " in r.stdout
    assert "D: 0 of" in r.stdout
