"""Invariants of Algorithm 1 checked on the vectorised oracle: exact round
trip of on-grid tensors, sign symmetry, power-of-two scale invariance,
permutation equivariance within a block, and the closed form of the block
holding the tensor maximum (s32 = amax / 2688 gives it the E4M3 scales 448 and
384, Algorithm 1)."""
import numpy as np
import pytest

from oracle import formats as F
from oracle import quant as Q
from workloads import bf16_bits_to_f32, f32_to_bf16_bits


def _ongrid(rng, rows, k, s32):
    """Blocks built from random codes on one grid, each block containing its
    grid maximum, so Algorithm 1 must pick exactly that scale back."""
    nb = rows * k // 16
    s8 = F.E4M3_VALUES[rng.integers(9, 120, nb)]
    fmt = rng.integers(0, 2, nb)
    mag = rng.integers(0, 8, (nb, 16))
    mag[np.arange(nb), rng.integers(0, 16, nb)] = 7
    v = np.where(fmt[:, None] == 1, F.I_GRID[mag], F.F_GRID[mag]) * s8[:, None]
    sgn = np.where(rng.random((nb, 16)) < 0.5, -1.0, 1.0)
    x = (sgn * v * s32).astype(np.float32).reshape(rows, k)
    bits = f32_to_bf16_bits(x)
    assert np.array_equal(bf16_bits_to_f32(bits), x)          # representable in bf16
    return bits, x


@pytest.mark.parametrize("s32", [1.0, 2.0 ** -7, 2.0 ** 5])
def test_round_trip_on_grid(s32):
    rng = np.random.default_rng(3)
    bits, x = _ongrid(rng, 32, 256, s32)
    q = Q.quantize(bits, s32=np.float32(s32))
    assert np.array_equal(Q.dequantize(q.codes, q.scales, q.s32), x)


def test_sign_symmetry():
    rng = np.random.default_rng(4)
    x = (rng.standard_t(3, (32, 128)) * 3).astype(np.float32)
    bits = f32_to_bf16_bits(x)
    q1 = Q.quantize(bits)
    q2 = Q.quantize(bits ^ np.uint16(0x8000))
    assert q1.s32 == q2.s32
    assert np.array_equal(q1.scales, q2.scales)
    assert np.array_equal(q1.codes ^ np.uint8(0x88), q2.codes)


@pytest.mark.parametrize("k", [-20, -3, 1, 9])
def test_power_of_two_scale_invariance(k):
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((16, 128)) * 0.7).astype(np.float32)
    bits = f32_to_bf16_bits(x)
    bits2 = f32_to_bf16_bits(x * np.float32(2.0 ** k))
    q1, q2 = Q.quantize(bits), Q.quantize(bits2)
    assert q2.s32 == np.float32(q1.s32 * np.float32(2.0 ** k))
    assert np.array_equal(q1.scales, q2.scales)
    assert np.array_equal(q1.codes, q2.codes)


def test_permutation_within_block():
    rng = np.random.default_rng(6)
    x = rng.laplace(0, 1, (8, 64)).astype(np.float32)
    bits = f32_to_bf16_bits(x)
    perm = rng.permutation(16)
    bits_p = bits.reshape(8, 4, 16)[:, :, perm].reshape(8, 64)
    q1, q2 = Q.quantize(bits), Q.quantize(bits_p)
    assert np.array_equal(q1.scales, q2.scales)
    n1 = Q.unpack_nibbles(q1.codes).reshape(8, 4, 16)[:, :, perm].reshape(8, 64)
    assert np.array_equal(n1, Q.unpack_nibbles(q2.codes))


@pytest.mark.parametrize("seed", range(5))
def test_amax_block_closed_form(seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_t(2, (16, 256)) * rng.uniform(1e-3, 1e3)).astype(np.float32)
    bits = f32_to_bf16_bits(x)
    q = Q.quantize(bits)
    xa = np.abs(bf16_bits_to_f32(bits))
    r, c = np.unravel_index(np.argmax(xa), xa.shape)
    b = c // 16
    assert q.s32 == np.float32(np.float32(xa.max()) / np.float32(2688))
    assert F.E4M3_VALUES[q.sf_code[r, b]] == 448 and F.E4M3_VALUES[q.si_code[r, b]] == 384
    assert q.scales[r, b] in (0x7E, 0xFC)
    nib = Q.unpack_nibbles(q.codes)[r, c]
    assert nib & 7 == 7


def test_t0_blocks_are_nvfp4():
    """Where Algorithm 1 keeps E2M1 (T = 0) the block is the NVFP4 encoding:
    E4M3 scale of block-max/6 and E2M1 codes (Sec. 2.1)."""
    rng = np.random.default_rng(8)
    x = rng.laplace(0, 1, (32, 128)).astype(np.float32)
    x.reshape(-1, 16)[:, 0] *= 30
    bits = f32_to_bf16_bits(x)
    q = Q.quantize(bits)
    t0 = q.t == 0
    assert t0.mean() > 0.5
    xb = np.abs(bf16_bits_to_f32(bits) / q.s32).astype(np.float32).reshape(32, 8, 16)
    s8 = F.E4M3_VALUES[F.e4m3_encode((xb.max(-1) / np.float32(6)).astype(np.float64))]
    y = (xb / s8[..., None].astype(np.float32)).astype(np.float64)
    codes = F.round_to_codebook(y, F.F_GRID)
    nib = Q.unpack_nibbles(q.codes).reshape(32, 8, 16) & 7
    assert np.array_equal(nib[t0], codes[t0])


def test_all_zero_and_negative_zero():
    bits = np.zeros((2, 32), np.uint16)
    bits[1, :16] = 0x8000
    q = Q.quantize(bits)
    assert q.s32 == 1.0
    assert q.scales.tolist() == [[0x80, 0x80], [0x80, 0x80]]
    assert q.codes[1, :8].tolist() == [0x88] * 8 and q.codes[0].tolist() == [0] * 16
    assert np.all(Q.dequantize(q.codes, q.scales, q.s32) == 0)
