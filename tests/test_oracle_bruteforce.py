"""Pins for the vectorised oracle (oracle.quant) against the brute-force
rational oracle (oracle.exact): nearest value by scanning every code of the
exact quotient, exact squared-error sums, and the literal Algorithm 1 choice.

Inputs: random blocks of several distributions, blocks whose elements sit on
or one fp32 ulp beside a rounding midpoint (tensor scales 1 +- k*2^-23 turn
exact bf16 midpoints into near-midpoints in the FP8 domain), and exhaustive
two-element blocks over a window of bf16 values."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import exact as E
from oracle import formats as F
from oracle import quant as Q
from workloads import f32_to_bf16_bits


def _compare(bits, s32=None):
    q = Q.quantize(bits, s32=s32)
    codes, scales, s = E.quantize(bits, s32=None if s32 is None else Fraction(float(np.float32(s32))))
    assert Fraction(float(q.s32)) == s
    np.testing.assert_array_equal(q.scales, np.array(scales, dtype=np.uint8))
    np.testing.assert_array_equal(q.codes, np.array(codes, dtype=np.uint8))
    return q


@pytest.mark.parametrize("dist", ["normal", "t3", "laplace_spike", "uniform", "lattice", "tiny_range"])
def test_random_blocks(dist):
    rng = np.random.default_rng(hash(dist) % 2**32)
    shape = (16, 64)
    if dist == "normal":
        x = rng.standard_normal(shape)
    elif dist == "t3":
        x = rng.standard_t(3, shape) * 7.3
    elif dist == "laplace_spike":
        x = rng.laplace(0, 1, shape)
        x.reshape(-1, 16)[np.arange(x.size // 16), rng.integers(0, 16, x.size // 16)] *= 40
    elif dist == "uniform":
        x = rng.uniform(-1, 1, shape) * 1e-3
    elif dist == "lattice":
        x = rng.integers(-7, 8, shape) * 0.375
    else:
        x = rng.standard_normal(shape) * np.where(rng.random((16, 1)) < 0.5, 1e-7, 1e3)
    bits = f32_to_bf16_bits(x.astype(np.float32))
    _compare(bits)
    _compare(bits, s32=np.float32(0.0173))


def test_near_midpoints():
    """X = mid * s8 exactly (bf16) and its bf16 neighbours, with tensor scales
    slightly off 1 so the FP8-domain values land within an fp32 ulp of a
    midpoint on either side, or exactly on it."""
    rows = []
    for s8 in F.E4M3_VALUES[40:120:7]:
        for grid, top in ((F.F_GRID, 6.0), (F.I_GRID, 7.0)):
            mids = (grid[:-1] + grid[1:]) / 2
            vals = [top * s8] + list(mids * s8)
            blk = np.zeros(16, np.float32)
            blk[:len(vals)] = vals
            rows.append(blk)
    x = np.stack(rows)
    bits = f32_to_bf16_bits(x)
    nb = np.where(bits != 0, bits + 1, bits).astype(np.uint16)     # next bf16 up (positive values)
    for b in (bits, nb):
        for s in (1.0, 1 + 2 ** -23, 1 - 2 ** -24, 1 + 3 * 2 ** -23, 1 - 3 * 2 ** -24):
            _compare(b, s32=np.float32(s))


def test_two_element_blocks_exhaustive_window():
    """Block = [a, b, 0, ...]: a over a few block maxima, b over every bf16
    pattern in [a/64, a] (bf16 bits are ordered like magnitudes)."""
    rows = []
    for a in (1.0, 6.0, 7.0, 2.71875, 413.0):
        abits = int(f32_to_bf16_bits(np.array([a], np.float32))[0])
        lo = int(f32_to_bf16_bits(np.array([a / 64], np.float32))[0])
        for bb in range(lo, abits + 1):
            r = np.zeros(16, np.uint16)
            r[0] = abits
            r[1] = bb
            rows.append(r)
    bits = np.stack(rows)
    _compare(bits, s32=np.float32(1.0))
    _compare(bits, s32=np.float32(0.8123))


def test_subnormal_scales_and_zero_blocks():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((4, 64)).astype(np.float32)
    x[0] *= 1e-5                       # block maxima far below the tensor max
    x[1] = 0.0
    x[2, :16] = -0.0
    x[3, 0] = 3000.0
    _compare(f32_to_bf16_bits(x))
