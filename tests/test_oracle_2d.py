"""Pins of the oracle's 2D (16x16-tile) weight quantization.

  * brute force: every tile through the rational oracle (Algorithm 1 on the
    256 tile elements, nearest code of the exact quotient, exact errors);
  * transposition: quantizing W^T gives the W^T layout of quantizing W, and
    the two layouts dequantize to exact transposes;
  * NVFP4 2D by construction (mode "e2m1"): E4M3(tile max / 6) through
    torch's float8_e4m3fn cast and nearest-even E2M1 codes from Table 1's
    grid, written out here;
  * a tile with one nonzero row is the 1D quantization of that row.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import workloads as W
from oracle import exact as E
from oracle import formats as F
from oracle import quant as Q


def _weight(seed, n=48, k=64):
    rng = np.random.default_rng(seed)
    w = rng.normal(0, 0.02, (n, k))
    w[rng.random((n, k)) < 0.01] *= 40
    w[:16, :16] = np.arange(256).reshape(16, 16) * 0.001      # a lattice-like tile
    w[16:32, 16:32] = 0.0                                       # an all-zero tile
    w[32:48, 32:48] = -0.0
    return W.f32_to_bf16_bits(w.astype(np.float32))


@pytest.mark.parametrize("mode", ["select", "e2m1", "e1m2"])
@pytest.mark.parametrize("seed,s32", [(0, None), (1, 0.001)])
def test_matches_bruteforce(mode, seed, s32):
    bits = _weight(seed)
    q = Q.quantize_2d(bits, s32=s32, mode=mode)
    s = Fraction(float(q.s32))
    nib = Q.unpack_nibbles(q.codes)
    n, k = bits.shape
    for a in range(n // 16):
        for b in range(k // 16):
            tile = bits[16 * a:16 * a + 16, 16 * b:16 * b + 16].reshape(-1)
            sb, nibs, _, _ = E.quantize_block(list(tile), s, mode)
            assert q.tile_scales[a, b] == sb, (a, b)
            assert np.array_equal(nib[16 * a:16 * a + 16, 16 * b:16 * b + 16].reshape(-1),
                                  np.array(nibs, np.uint8)), (a, b)


@pytest.mark.parametrize("seed", [2, 3])
def test_transpose_consistency(seed):
    bits = W.adversarial(seed, 64, 96)
    q = Q.quantize_2d(bits)
    qt = Q.quantize_2d(np.ascontiguousarray(bits.T))
    assert qt.s32 == q.s32
    assert np.array_equal(qt.codes, q.codes_t) and np.array_equal(qt.scales, q.scales_t)
    assert np.array_equal(qt.codes_t, q.codes) and np.array_equal(qt.scales_t, q.scales)
    d = Q.dequantize(q.codes, q.scales, q.s32)
    dt = Q.dequantize(q.codes_t, q.scales_t, q.s32)
    assert np.array_equal(d, dt.T)


def test_nvfp4_2d_by_construction():
    bits = _weight(4, 64, 80)
    q = Q.quantize_2d(bits, mode="e2m1")
    x = (W.bf16_bits_to_f32(bits) / q.s32).astype(np.float32)
    n, k = bits.shape
    tiles = np.abs(x).reshape(n // 16, 16, k // 16, 16).transpose(0, 2, 1, 3)
    bm = tiles.max(axis=(-1, -2))
    cand = torch.from_numpy((bm / np.float32(6)).astype(np.float32))
    code = cand.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(q.tile_scales, code)
    s8 = cand.to(torch.float8_e4m3fn).to(torch.float32).numpy()
    grid = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6])
    with np.errstate(divide="ignore", invalid="ignore"):
        y = np.where(s8[..., None, None] > 0, tiles / s8[..., None, None], 0).astype(np.float32)
    dist = np.abs(y.astype(np.float64)[..., None] - grid)
    best = dist.min(-1, keepdims=True)
    ties = (dist == best)
    idx = np.where(ties & (np.arange(8) % 2 == 0), np.arange(8), 99).min(-1)
    idx = np.where(idx == 99, np.where(ties, np.arange(8), 99).min(-1), idx)
    mag = Q.unpack_nibbles(q.codes) & 7
    want = idx.transpose(0, 2, 1, 3).reshape(n, k)
    assert np.array_equal(mag, want)


def test_single_row_tiles_equal_1d():
    rng = np.random.default_rng(5)
    n, k = 64, 128
    w = np.zeros((n, k), np.float32)
    for a in range(n // 16):
        for b in range(k // 16):
            i = int(rng.integers(0, 16))
            w[16 * a + i, 16 * b:16 * b + 16] = rng.standard_t(3, 16)
    bits = W.f32_to_bf16_bits(w)
    q2 = Q.quantize_2d(bits)
    q1 = Q.quantize(bits)
    assert q2.s32 == q1.s32
    assert np.array_equal(q2.codes, q1.codes)
    nz = np.abs(w).reshape(n, k // 16, 16).max(-1) > 0
    assert np.array_equal(q2.scales[nz], q1.scales[nz])


def test_layout_repeats_tile_bytes():
    bits = _weight(6, 32, 48)
    q = Q.quantize_2d(bits)
    for a in range(2):
        for b in range(3):
            assert np.all(q.scales[16 * a:16 * a + 16, b] == q.tile_scales[a, b])
            assert np.all(q.scales_t[16 * b:16 * b + 16, a] == q.tile_scales[a, b])
