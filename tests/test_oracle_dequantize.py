"""Pins for oracle.quant.dequantize / dequantize_exact (App. B.2-B.3 decode).

An element of a MixFP4 tensor stands for s32 * s8 * v(code, T) * sign.  The
product s8 * v is exact (at most 4 + 3 significant bits), so the fp32 output
is that real number rounded once.  These tests check that rounding against
the rational brute force of ``oracle.exact`` (its own codebooks from the
value equation, its own IEEE binary32 rounding written from the definition)
at tensor scales that are NOT powers of two, where a second rounding (for
example of s32 * s8 before the multiplication by v) changes the result.
"""
from fractions import Fraction

import numpy as np

from oracle import exact as E
from oracle import quant as Q

# Non-power-of-two tensor scales (fp32 values): an adversarial workload's s32,
# a short decimal, one ulp above 1, a huge and a tiny one whose products reach
# the ends of the fp32 range (subnormal outputs included).
S32_CASES = [np.float32(11.142858), np.float32(0.37), np.float32(1.0 + 2.0 ** -23),
             np.float32(3.0 * 2.0 ** 100 + 2.0 ** 80), np.float32(5.0 * 2.0 ** -140)]


def _codes_and_scales(rows: int = 8, k: int = 256, seed: int = 7):
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 256, (rows, k // 2), dtype=np.uint8)
    # every finite scale byte, both T values (0x7F / 0xFF are E4M3 NaN)
    sb = rng.integers(0, 0x7F, (rows, k // 16), dtype=np.uint8)
    t = rng.integers(0, 2, (rows, k // 16), dtype=np.uint8)
    sb[0, :] = np.arange(k // 16, dtype=np.uint8) * 8 % 0x7F
    return codes, (sb | (t << 7)).astype(np.uint8)


def _rational_decode(codes, scales, s32):
    """round_f32(decode_value * s32) element by element, as Fractions."""
    rows, half = codes.shape
    out = np.empty((rows, 2 * half), dtype=object)
    s = Fraction(float(s32))
    for r in range(rows):
        for j in range(2 * half):
            byte = int(codes[r, j // 2])
            nib = byte & 0x0F if j % 2 == 0 else byte >> 4
            out[r, j] = E.decode_value(nib, int(scales[r, j // 16])) * s
    return out


def dequantize_pins_pass() -> bool:
    codes, scales = _codes_and_scales()
    for s32 in S32_CASES:
        exact = _rational_decode(codes, scales, s32)
        got = Q.dequantize(codes, scales, s32)
        got_exact = Q.dequantize_exact(codes, scales, s32)
        for idx in np.ndindex(exact.shape):
            want = E.round_f32(exact[idx])
            if Fraction(float(got[idx])) != want:
                return False
            if Fraction(float(got_exact[idx])) != exact[idx]:
                return False
    return True


def test_dequantize_rounds_once_at_non_power_of_two_scales():
    assert dequantize_pins_pass()


def test_dequantize_scale_none_is_the_fp8_domain():
    codes, scales = _codes_and_scales(rows=2, k=64, seed=3)
    d = Q.dequantize(codes, scales, None)
    exact = _rational_decode(codes, scales, np.float32(1.0))
    for idx in np.ndindex(exact.shape):
        assert Fraction(float(d[idx])) == exact[idx]      # s8 * v is exact in fp32


def test_cases_separate_one_rounding_from_two():
    """The pin only means something if rounding s32 * s8 first would change
    some outputs at these scales; count such elements from the rationals."""
    codes, scales = _codes_and_scales()
    differ = 0
    for s32 in S32_CASES:
        s = Fraction(float(s32))
        nib = Q.unpack_nibbles(codes)
        for r in range(codes.shape[0]):
            for j in range(codes.shape[1] * 2):
                sb = int(scales[r, j // 16])
                unit = E.decode_value(int(nib[r, j]), sb)
                s8 = E.E4M3[sb & 0x7F][1]
                if s8 == 0:
                    continue
                once = E.round_f32(unit * s)
                twice = E.round_f32(E.round_f32(s8 * s) * (unit / s8))
                differ += once != twice
    assert differ > 100
