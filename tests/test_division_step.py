"""The quantizer divides in fp32 without a divide instruction: x = X / s32
with one multiply and two fmas on a correctly rounded reciprocal, and the
quotients by the block scales (and by 6 and 7) with a multiply and one fma
on a two-term reciprocal.  tests/division_step.c proves on the CPU,
exhaustively over the operand mantissas the kernel can see, that both give
the IEEE quotient bit for bit, and that zeros keep their sign."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))

# Every (s32 in [1, 2), bf16 X in [1, 2)) pair, as fp32 bits, on which the
# two-term step misses the IEEE quotient X / s32 (part E of division_step.c):
# the quantizer's launch-time check sends these tensor scales (at any
# exponent) to Markstein's step.  The GPU tests drive that fallback with them.
FALLBACK_PAIRS = [
    (0x3F9CDFAB, 0x3F890000), (0x3FBC49AB, 0x3FEE0000), (0x3FD0AB43, 0x3FC70000),
    (0x3FD2D00F, 0x3FB10000), (0x3FDB4E6B, 0x3FCB0000), (0x3FE190F3, 0x3FB20000),
    (0x3FE241EF, 0x3FD90000), (0x3FE5AE9F, 0x3FEB0000), (0x3FEB3CA3, 0x3FDB0000),
    (0x3FF28673, 0x3FCB0000), (0x3FF92863, 0x3FF40000),
]


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
    census = sorted((int(a, 16), int(b, 16)) for a, b in
                    re.findall(r"^E s32 0x([0-9a-f]+) X 0x([0-9a-f]+)$", r.stdout, re.M))
    assert census == sorted(FALLBACK_PAIRS)
