"""Pins of the oracle's 4/6 mode (the candidate set {E2M1(6), E2M1(4)} the
paper compares MixFP4 against, Sec. 2.3 and Sec. 4.2): E2M1 codes under the
block scale E4M3(max/6) or E4M3(max/4), whichever has the smaller squared
error, ties keeping /6; T = 0 everywhere (plain NVFP4).

  * brute force: the rational oracle in the same mode;
  * by construction: both candidates written out here (torch's
    float8_e4m3fn cast for the scales, Table 1's E2M1 grid with nearest /
    ties-to-even-code for the codes, exact rational errors), the choice
    checked;
  * invariants: T = 0; the squared error never exceeds NVFP4's; where the
    /6 candidate is kept the block equals NVFP4's ("e2m1" mode).
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import workloads as W
from oracle import exact as E
from oracle import quant as Q


def _x(seed, rows=12, k=64):
    rng = np.random.default_rng(seed)
    x = rng.laplace(0, 1, (rows, k))
    x.reshape(-1, 16)[::3, 5] *= 30
    x[0, :16] = np.arange(16) * 0.25
    x[1, :16] = 0.0
    x[2, :16] = [4, 3, 2, 1.5, 1, 0.5, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0]
    # ties at s32 = 1: both candidates exact (6 = 1 * 6 = 1.5 * 4; 3 = .5 * 6 =
    # .75 * 4 and 1.5 = .5 * 3 = .75 * 2), so /6 must be kept
    x[3, :16] = 0.0
    x[3, 0] = 6.0
    x[3, 16:32] = 0.0
    x[3, 16:18] = [3.0, -1.5]
    return W.f32_to_bf16_bits(x.astype(np.float32))


@pytest.mark.parametrize("seed,s32", [(0, None), (1, 0.25), (2, 1.0)])
def test_matches_bruteforce(seed, s32):
    bits = _x(seed)
    q = Q.quantize(bits, s32=s32, mode="four_six")
    codes, scales, s = E.quantize(bits, s32=None if s32 is None else Fraction(float(np.float32(s32))),
                                  mode="four_six")
    assert np.array_equal(q.scales, np.array(scales, np.uint8))
    assert np.array_equal(q.codes, np.array(codes, np.uint8))


def _candidate(xb, divisor):
    """E4M3(max/divisor) by torch's cast and nearest-even E2M1 codes of the
    exact quotients; returns (scale code, scale, codes, exact SSE)."""
    grid = [Fraction(v) for v in ("0", "0.5", "1", "1.5", "2", "3", "4", "6")]
    bm = np.float32(np.abs(xb).max())
    # E4M3 saturates at 448 (torch's cast would give NaN above it)
    cand = torch.tensor([min(np.float32(bm / np.float32(divisor)), np.float32(448.0))])
    f8 = cand.to(torch.float8_e4m3fn)
    code = int(f8.view(torch.uint8)[0])
    s8 = Fraction(float(f8.to(torch.float32)[0]))
    codes, sse = [], Fraction(0)
    for v in xb:
        a = abs(Fraction(float(v)))
        if s8 == 0:
            c = 0
        else:
            q = a / s8
            d = [abs(q - g) for g in grid]
            best = min(d)
            ties = [i for i, dv in enumerate(d) if dv == best]
            c = next((i for i in ties if i % 2 == 0), ties[0])
        codes.append(c)
        sse += (a - grid[c] * s8) ** 2
    return code, codes, sse


def test_by_construction():
    bits = _x(3)
    q = Q.quantize(bits, mode="four_six")
    x = (W.bf16_bits_to_f32(bits) / q.s32).astype(np.float32)
    nib = Q.unpack_nibbles(q.codes)
    rows, k = bits.shape
    for r in range(rows):
        for b in range(k // 16):
            xb = x[r, 16 * b:16 * b + 16]
            c6, q6, e6 = _candidate(xb, 6)
            c4, q4, e4 = _candidate(xb, 4)
            use4 = e4 < e6
            assert q.scales[r, b] == (c4 if use4 else c6)
            assert list(nib[r, 16 * b:16 * b + 16] & 7) == (q4 if use4 else q6)


def test_invariants():
    bits = _x(4, 32, 128)
    q46 = Q.quantize(bits, mode="four_six")
    qnv = Q.quantize(bits, mode="e2m1")
    assert np.all(q46.scales >> 7 == 0)
    d46 = Q.dequantize_exact(q46.codes, q46.scales, q46.s32)
    dnv = Q.dequantize_exact(qnv.codes, qnv.scales, qnv.s32)
    x = W.bf16_bits_to_f32(bits).astype(np.float64)
    e46 = ((x - d46) ** 2).reshape(32, -1, 16).sum(-1)
    env = ((x - dnv) ** 2).reshape(32, -1, 16).sum(-1)
    assert np.all(e46 <= env * (1 + 1e-12) + 1e-300)
    kept6 = q46.scales == qnv.scales
    n46, nnv = Q.unpack_nibbles(q46.codes), Q.unpack_nibbles(qnv.codes)
    same = (n46 == nnv).reshape(32, -1, 16).all(-1)
    assert np.all(same[kept6])
    assert (~kept6).any() and kept6.any()


def test_ties_keep_six():
    bits = _x(2)
    q = Q.quantize(bits, s32=1.0, mode="four_six")
    assert q.scales[3, 0] == 0x38 and q.scales[3, 1] == 0x30      # E4M3 1.0 and 0.5
