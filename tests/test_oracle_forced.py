"""Pins for the oracle's forced-format modes: "e2m1" keeps the E2M1 branch of
Algorithm 1 for every block (NVFP4, Sec. 2.1) and "e1m2" the E1M2 (INT4)
branch, with the same tensor-scale rule.

- brute force: the vectorised oracle equals the rational oracle (nearest
  value by scanning every code of the exact quotient) in both modes;
- NVFP4 by construction: "e2m1" equals an E4M3(max/6) scale with
  round-to-nearest-even E2M1 codes, written out here from Table 1's grid;
- INT4 by construction: "e1m2" equals an E4M3(max/7) scale with
  round-half-even integer codes clamped at 7;
- consistency: where MixFP4 picks a format, the forced mode of that format
  gives the same block; T records the forced branch everywhere."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import exact as E
from oracle import formats as F
from oracle import quant as Q
from workloads import adversarial, bf16_bits_to_f32, f32_to_bf16_bits


def _blocks(seed):
    rng = np.random.default_rng(seed)
    x = rng.laplace(0, 1, (8, 64))
    x.reshape(-1, 16)[:, 3] *= 25
    x[0, :16] = np.arange(16) * 0.5          # exactly on the grids
    x[1, :16] = 0.0
    return f32_to_bf16_bits(x.astype(np.float32))


@pytest.mark.parametrize("mode", ["e2m1", "e1m2"])
@pytest.mark.parametrize("seed,s32", [(0, None), (1, 0.37), (2, 1.0)])
def test_forced_matches_bruteforce(mode, seed, s32):
    bits = _blocks(seed)
    q = Q.quantize(bits, s32=s32, mode=mode)
    codes, scales, s = E.quantize(bits, s32=None if s32 is None else Fraction(float(np.float32(s32))),
                                  mode=mode)
    assert Fraction(float(q.s32)) == s
    np.testing.assert_array_equal(q.scales, np.array(scales, dtype=np.uint8))
    np.testing.assert_array_equal(q.codes, np.array(codes, dtype=np.uint8))


def _by_construction(bits, divisor, grid):
    rows, k = bits.shape
    q = Q.quantize(bits)                     # only for s32 (Algorithm 1's first step)
    x = (bf16_bits_to_f32(bits) / q.s32).astype(np.float32).reshape(rows, k // 16, 16)
    bm = np.abs(x).max(-1)
    code = F.e4m3_encode((bm / np.float32(divisor)).astype(np.float32).astype(np.float64))
    s8 = F.E4M3_VALUES[code].astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        y = np.where(s8[..., None] > 0, np.abs(x) / s8[..., None], 0).astype(np.float64)
    # nearest grid value, ties to the even index, written out directly
    dist = np.abs(y[..., None] - grid)
    best = dist.min(-1, keepdims=True)
    cand = np.where(dist == best, np.arange(len(grid)), 99)
    idx = np.where((cand % 2 == 0) & (cand != 99), cand, 99).min(-1)
    idx = np.where(idx == 99, cand.min(-1), idx)
    return code, idx


def test_e2m1_mode_is_nvfp4():
    bits = adversarial(31, 12, 96)
    q = Q.quantize(bits, mode="e2m1")
    code, idx = _by_construction(bits, 6, F.F_GRID)
    assert np.all(q.scales >> 7 == 0)
    np.testing.assert_array_equal(q.scales & 0x7F, code)
    np.testing.assert_array_equal(Q.unpack_nibbles(q.codes).reshape(idx.shape) & 7, idx)


def test_e1m2_mode_is_int4():
    bits = adversarial(32, 12, 96)
    q = Q.quantize(bits, mode="e1m2")
    code, idx = _by_construction(bits, 7, F.I_GRID)
    assert np.all(q.scales >> 7 == 1)
    np.testing.assert_array_equal(q.scales & 0x7F, code)
    np.testing.assert_array_equal(Q.unpack_nibbles(q.codes).reshape(idx.shape) & 7, idx)


def test_forced_modes_agree_with_selection():
    bits = adversarial(33, 40, 128)
    sel = Q.quantize(bits)
    f = Q.quantize(bits, mode="e2m1")
    i = Q.quantize(bits, mode="e1m2")
    nb = bits.shape[1] // 16
    cs = Q.unpack_nibbles(sel.codes).reshape(-1, nb, 16)
    cf = Q.unpack_nibbles(f.codes).reshape(-1, nb, 16)
    ci = Q.unpack_nibbles(i.codes).reshape(-1, nb, 16)
    t = sel.t.astype(bool)
    np.testing.assert_array_equal(sel.scales[~t], f.scales[~t])
    np.testing.assert_array_equal(sel.scales[t], i.scales[t])
    np.testing.assert_array_equal(cs[~t], cf[~t])
    np.testing.assert_array_equal(cs[t], ci[t])
    # signs are X's in every mode
    np.testing.assert_array_equal(cf & 8, cs & 8)
    np.testing.assert_array_equal(ci & 8, cs & 8)
