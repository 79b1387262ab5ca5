"""Block-diagonal (random) Hadamard transform of a bf16 matrix along K.

TEST INFRASTRUCTURE (oracle); see ``oracle/__init__``.

The paper rotates tensors with a random Hadamard transform before MixFP4
quantization: in the training recipe of Sec. 3.2 (Fig. 7, the inputs of the
weight-gradient GEMM) and Sec. 4.3, and in the "+RHT" PTQ rows of Table 3
(Sec. 4.2), where Hadamard mixing spreads outliers across a block of
coordinates (Sec. 1, Sec. 2.2).  The transform is orthonormal and acts on
consecutive blocks of b coordinates along the reduction dimension:

    y[c*b + j] = sum_i  s_i * x[c*b + i] * H_b[i, j] / sqrt(b)

with H_b the Sylvester Hadamard matrix (H_1 = [1], H_2n = [[H_n, H_n],
[H_n, -H_n]]; entry (i, j) is (-1)^popcount(i & j)) and s a vector of b signs
(all +1 for the plain transform; random for the RHT).

Readings (the paper does not fix them; listed in the design notes):
  * input and output are bf16; each output is the exact value above rounded
    once to bf16, to nearest with ties to even (an overflow becomes Inf);
  * the signs multiply the inputs (y = (s . x) H / sqrt(b)), one sign
    vector for every block of every row;
  * b is a power of two from 16 to 256 and divides K.

Exactness here: the block sums are a float64 matrix product, exact when the
block is certified (every nonzero input is a multiple of 2^u and the absolute
sum stays below 2^(u+53)); elements of other blocks are summed with
rationals.  For b a power of 4 the division by
sqrt(b) is exact; otherwise the float64 quotient is within 2^-51 of the exact
one, and every element whose bf16 rounding is not settled by that bound is
decided exactly by comparing squares of integers.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

BLOCKS = (16, 32, 64, 128, 256)
BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127


def sylvester(b: int) -> np.ndarray:
    """H_b by the doubling construction (int64 entries +-1)."""
    assert b >= 1 and b & (b - 1) == 0
    h = np.ones((1, 1), dtype=np.int64)
    while h.shape[0] < b:
        h = np.block([[h, h], [h, -h]])
    return h


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32) \
        .astype(np.float64)


def round_to_bf16(y: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (nearest, ties to even, gradual underflow
    with spacing 2^-133, Inf beyond the largest finite value after rounding);
    returns bf16 bit patterns.  Written from the format: 8 significant bits
    in the binade of y, at least the spacing of the smallest normal binade."""
    y = np.asarray(y, dtype=np.float64)
    a = np.abs(y)
    _, e = np.frexp(a)                                  # a = m * 2^e, m in [0.5, 1)
    e = np.maximum(e - 1, -126)                          # binade exponent, subnormals share -126
    ulp = np.ldexp(1.0, (e - 7).astype(np.int64))
    n = np.rint(a / ulp)                                 # exact quotient, half to even
    r = n * ulp
    r = np.where(r > BF16_MAX, np.inf, r)
    r = np.where(np.signbit(y), -r, r)
    return (r.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _certified_blocks(x: np.ndarray) -> np.ndarray:
    """Mask of Hadamard blocks (rows of ``x`` [n, b], exact float64 values)
    whose sums sum_i +-x_i are exact in float64 in any order: every nonzero
    x_i is a multiple of 2^u (u = the lowest set bit over the block) and
    sum |x_i| < 2^(u + 53), so every partial sum is a multiple of 2^u below
    2^(u + 53) and representable."""
    nz = x != 0
    m, e = np.frexp(x)
    mi = np.abs(np.ldexp(m, 53)).astype(np.int64)
    low = mi & (-mi)
    lowexp = np.where(nz, e.astype(np.float64) - 53.0 + np.log2(np.maximum(low, 1).astype(np.float64)),
                      np.inf)
    u = lowexp.min(axis=-1)
    total = np.abs(x).sum(axis=-1) * (1.0 + 2.0 ** -40)
    return np.isinf(u) | (total < np.ldexp(1.0, np.clip(u + 53, -1074, 1023).astype(np.int64)))


def bf16_bits_value(bits: int) -> Fraction:
    """Exact magnitude of bf16 bits (sign ignored); the pattern 0x7F80 reads
    as 2^128, the value one step above the largest finite bf16, which places
    the overflow threshold at the midpoint like any other."""
    e, m = (bits >> 7) & 0xFF, bits & 0x7F
    if e == 0:
        return Fraction(m) * Fraction(2) ** -133
    return Fraction(128 + m) * Fraction(2) ** (e - 134)


def _round_exact(v2: Fraction, guess: int) -> int:
    """bf16 magnitude bits of RNE(v) given v^2 = ``v2`` (exact, v > 0) and a
    float64-based guess within one step: move the guess while v lies beyond
    one of its rounding midpoints.  v = S / (2^m sqrt 2) with S != 0 is
    irrational, so it is never equal to a midpoint; a dyadic v (power-of-4
    blocks) is handled with the even rule at a midpoint."""
    bits = guess & 0x7FFF
    for _ in range(4):
        val = bf16_bits_value(bits)
        mid_hi = (val + bf16_bits_value(bits + 1)) / 2
        mid_lo = (val + bf16_bits_value(bits - 1)) / 2 if bits else Fraction(0)
        if v2 > mid_hi * mid_hi or (v2 == mid_hi * mid_hi and bits % 2 == 1):
            bits += 1
        elif bits and (v2 < mid_lo * mid_lo or (v2 == mid_lo * mid_lo and bits % 2 == 1)):
            bits -= 1
        else:
            break
        if bits >= 0x7F80:
            return 0x7F80
    return bits


def _exact_element(terms: np.ndarray, level: int) -> int:
    """bf16 bits of one output from its b exact terms, all in rationals."""
    S = Fraction(0)
    for t in terms:
        S += Fraction(float(t))
    if S == 0:
        return 0
    v2 = S * S / 2 ** level                              # (S / sqrt(b))^2
    guess = float(abs(S)) / math.sqrt(2.0 ** level)
    g = int(round_to_bf16(np.array([guess]))[0])
    bits = _round_exact(v2, g)
    return bits | (0x8000 if S < 0 else 0)


def hadamard(x_bits: np.ndarray, b: int, signs=None) -> np.ndarray:
    """The block-diagonal transform of a bf16 matrix (uint16 [rows, K]) with
    blocks of ``b`` and optional signs (length-b array of +-1); returns bf16
    bit patterns [rows, K], each the exact result rounded once (an exactly
    zero result is +0)."""
    assert b in BLOCKS
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    rows, k = x_bits.shape
    assert k % b == 0
    s = np.ones(b, dtype=np.int64) if signs is None else np.asarray(signs, dtype=np.int64)
    assert s.shape == (b,) and np.all(np.abs(s) == 1)
    if x_bits.size == 0:
        return x_bits.copy()
    level = int(round(math.log2(b)))
    H = sylvester(b).astype(np.float64)
    x = bf16_bits_to_f64(x_bits).reshape(-1, b) * s[None, :]           # exact (sign flips)
    # S[c, j] = sum_i x[c, i] H[i, j]: a float64 product, exact for certified blocks
    S = x @ H
    ok = np.repeat(_certified_blocks(x)[:, None], b, axis=1)
    v = S / math.sqrt(2.0 ** level)                      # exact for even level, else within 2^-52
    res = round_to_bf16(v)
    if level % 2:
        # settled when both ends of the error interval round alike
        ok &= round_to_bf16(v * (1.0 - 2.0 ** -50)) == round_to_bf16(v * (1.0 + 2.0 ** -50))
    res = np.where(S == 0, np.uint16(0), res)
    for c, j in np.argwhere(~ok):
        res[c, j] = _exact_element(x[c] * H[:, j], level)
    return res.reshape(rows, k)
