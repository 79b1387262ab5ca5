"""Pins of the block-diagonal Hadamard transform in the oracle.

  * the Sylvester matrix against scipy's and H H^T = b I;
  * unit vectors map to a row of H / sqrt(b) (hand-derived bf16 values);
  * an independent route: the fast Walsh-Hadamard butterflies in rationals,
    rounded to bf16 through 120-digit decimal arithmetic;
  * elements built to lie within 2^-60 of a bf16 rounding midpoint;
  * involution on integer data, sign vectors, overflow, signed zeros.
"""
import decimal
import math
from fractions import Fraction

import numpy as np
import pytest
import scipy.linalg

import workloads as W
from oracle import hadamard as HD

decimal.getcontext().prec = 120


def test_sylvester_matches_scipy_and_is_orthogonal():
    for b in HD.BLOCKS:
        h = HD.sylvester(b)
        assert np.array_equal(h, scipy.linalg.hadamard(b))
        assert np.array_equal(h @ h.T, b * np.eye(b, dtype=np.int64))


def test_unit_vectors():
    """e_i maps to row i of H / sqrt(b).  By hand: 1/4 = 0x3E80 for b = 16;
    1/(8 sqrt 2) = 0.0883883... = 1.41421 * 2^-4, whose 8-bit significand
    rounds to 181/128, bits 0x3DB5, for b = 128."""
    for b, mag in ((16, 0x3E80), (128, 0x3DB5), (64, 0x3E00), (256, 0x3D80)):
        h = HD.sylvester(b)
        for i in (0, 3, b - 1):
            x = np.zeros((1, b), np.uint16)
            x[0, i] = 0x3F80
            y = HD.hadamard(x, b)[0]
            want = np.where(h[i] > 0, mag, mag | 0x8000).astype(np.uint16)
            assert np.array_equal(y, want), (b, i)


def _dec_round_bf16(S: Fraction, b: int) -> int:
    """RNE to bf16 of S / sqrt(b) through 120-digit decimals (independent of
    the oracle's rounding)."""
    if S == 0:
        return 0
    D = decimal.Decimal
    v = abs(D(S.numerator) / D(S.denominator)) / D(b).sqrt()
    e = 0
    while D(2) ** e > v:
        e -= 1
    while D(2) ** (e + 1) <= v:
        e += 1
    e = max(e, -126)
    q = v / (D(2) ** (e - 7))
    n = int(q.to_integral_value(rounding=decimal.ROUND_FLOOR))
    rem = q - n
    if rem > D("0.5") or (rem == D("0.5") and n % 2 == 1):
        n += 1
    val = n * Fraction(2) ** (e - 7)
    if val > Fraction(HD.BF16_MAX):
        bits = 0x7F80
    else:
        bits = int(np.array([float(val)], np.float32).view(np.uint32)[0] >> 16)
    return bits | (0x8000 if S < 0 else 0)


def _fwht_rational(vals):
    """Butterfly recursion: (a, b) -> (a + b, a - b) at strides 1, 2, 4, ..."""
    v = list(vals)
    h = 1
    while h < len(v):
        for i in range(0, len(v), 2 * h):
            for j in range(i, i + h):
                a, c = v[j], v[j + h]
                v[j], v[j + h] = a + c, a - c
        h *= 2
    return v


def _independent(bits, b, signs=None):
    rows, k = bits.shape
    x = HD.bf16_bits_to_f64(bits)
    s = [1] * b if signs is None else [int(t) for t in signs]
    out = np.zeros((rows, k), np.uint16)
    for r in range(rows):
        for c in range(0, k, b):
            v = _fwht_rational([Fraction(float(x[r, c + i])) * s[i] for i in range(b)])
            for j in range(b):
                out[r, c + j] = _dec_round_bf16(v[j], b)
    return out


@pytest.mark.parametrize("b", HD.BLOCKS)
def test_matches_rational_butterflies(b):
    rng = np.random.default_rng(b)
    x = rng.standard_t(3, (2, 2 * b)).astype(np.float32)
    x[0, :b // 2] *= np.float32(2.0 ** 60)           # wide exponent spread: rational sums
    x[1, 3] = 1e-30
    bits = W.f32_to_bf16_bits(x)
    signs = rng.choice([-1, 1], size=b)
    assert np.array_equal(HD.hadamard(bits, b), _independent(bits, b))
    assert np.array_equal(HD.hadamard(bits, b, signs), _independent(bits, b, signs))


def _split_bf16(S: int, pieces: int):
    """Write the integer S as a sum of bf16 values (8 significant bits each)."""
    out, rest = [], S
    for _ in range(pieces):
        if rest == 0:
            break
        e = abs(rest).bit_length() - 8
        part = (abs(rest) >> max(e, 0)) << max(e, 0)
        part = part if rest > 0 else -part
        out.append(part)
        rest -= part
    assert rest == 0
    return out


@pytest.mark.parametrize("b", [32, 128])
def test_near_midpoint_elements(b):
    """S chosen with S / sqrt(b) within ~2^-60 (relative) of a bf16 midpoint:
    float64 cannot settle the rounding; the exact decision must agree with
    the decimal one."""
    got_lo = got_hi = 0
    for mant in range(129, 200, 7):
        for side in (-1, 1):
            mid = Fraction(2 * mant + 1, 2) * Fraction(2) ** -7       # midpoint in [1, 2)
            target = mid * Fraction(2) ** 20
            approx = decimal.Decimal(target.numerator) / decimal.Decimal(target.denominator) \
                * decimal.Decimal(b).sqrt()
            S = int(approx.to_integral_value(rounding=decimal.ROUND_FLOOR)) + (1 if side > 0 else 0)
            parts = _split_bf16(S, 8)
            x = np.zeros((1, b), np.float32)
            x[0, :len(parts)] = np.array(parts, np.float64).astype(np.float32)
            assert sum(Fraction(float(p)) for p in x[0]) == S
            bits = W.f32_to_bf16_bits(x)
            y = HD.hadamard(bits, b)[0, 0]
            want = _dec_round_bf16(Fraction(S), b)
            assert y == want, (mant, side, hex(y), hex(want))
            got_lo += side < 0
            got_hi += side > 0
    assert got_lo and got_hi


def test_involution_on_integers():
    """For b a power of 4 and small integer data every step is exact, so the
    transform applied twice returns the input."""
    rng = np.random.default_rng(1)
    for b in (16, 64, 256):
        x = rng.integers(-8, 9, (4, 2 * b)).astype(np.float32)
        bits = W.f32_to_bf16_bits(x)
        y = HD.hadamard(bits, b)
        yy = HD.hadamard(y, b)
        back = HD.bf16_bits_to_f64(yy)
        assert np.array_equal(back, x.astype(np.float64))


def test_signs_act_on_inputs():
    rng = np.random.default_rng(2)
    b = 128
    x = rng.standard_normal((3, 256)).astype(np.float32)
    bits = W.f32_to_bf16_bits(x)
    s = rng.choice([-1, 1], size=b)
    flipped = W.f32_to_bf16_bits((x.reshape(-1, b) * s).reshape(x.shape).astype(np.float32))
    assert np.array_equal(HD.hadamard(bits, b, s), HD.hadamard(flipped, b))
    neg = HD.hadamard(bits, b, -np.ones(b, int))
    pos = HD.hadamard(bits, b)
    nz = (pos & 0x7FFF) != 0
    assert np.array_equal(neg[nz], pos[nz] ^ 0x8000)


def test_overflow_and_zeros():
    b = 16
    x = np.zeros((2, b), np.uint16)
    x[0, :] = 0x7F7F                                  # largest finite bf16
    x[1, :] = 0x8000                                  # -0
    y = HD.hadamard(x, b)
    assert y[0, 0] == 0x7F80                          # 16 max / 4 = 4 max -> Inf
    assert np.all(y[0, 1:] == 0)                      # exact zeros are +0
    assert np.all(y[1] == 0)


def test_subnormal_outputs():
    b = 32
    x = np.zeros((1, b), np.float64)
    x[0, :5] = [2.0 ** -130, 3 * 2.0 ** -133, -2.0 ** -128, 2.0 ** -131, 5 * 2.0 ** -133]
    bits = W.f32_to_bf16_bits(x.astype(np.float32))
    assert np.array_equal(HD.hadamard(bits, b), _independent(bits, b))
