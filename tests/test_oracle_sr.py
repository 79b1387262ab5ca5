"""Pins of the stochastic-rounding quantizer in the oracle (App. D) and of the
Philox4x32-10 draws it uses.

  * the generator against its published known-answer vectors;
  * hand-worked single roundings (tests/golden/sr_handworked.txt);
  * the INT4 branch against App. D's formula written out literally
    (clamp(round(q + eps - 1/2), -7, 7) on the signed quotient);
  * the E2M1 branch against the same formula on each uniform piece of the
    E2M1 grid ([0, 2) step 1/2, [2, 4) step 1, [4, 6] step 2);
  * the brute-force rational quantizer with the same draws;
  * unbiasedness over the 256 draws;
  * scales and format bits unchanged from round-to-nearest.
"""
import numpy as np
import pytest

import workloads as W
from oracle import exact as E
from oracle import formats as F
from oracle import philox as P
from oracle import quant as Q
from tests._golden import philox_kat, sr_handworked


def test_philox_known_answers():
    for v in philox_kat():
        got = P.philox4x32(np.array(v["counter"], np.uint64), np.array(v["key"], np.uint64),
                           rounds=v["rounds"])
        assert [int(w) for w in got] == v["out"], v


def test_block_bytes_layout():
    """Block g of a [rows, K] tensor uses counter (g lo, g hi, offset lo,
    offset hi); element j takes byte j % 4 of word j // 4."""
    rows, k, seed, offset = 3, 96, 0x1234567890ABCDEF, (7 << 32) | 5
    u = P.block_bytes(rows, k, seed, offset)
    nb = k // 16
    for r in range(rows):
        for kb in range(nb):
            g = r * nb + kb
            w = P.philox4x32(np.array([g, 0, 5, 7], np.uint64),
                             np.array([seed & 0xFFFFFFFF, seed >> 32], np.uint64))
            for j in range(16):
                assert u[r, kb * 16 + j] == (int(w[j // 4]) >> (8 * (j % 4))) & 0xFF
    assert not np.array_equal(u, P.block_bytes(rows, k, seed, offset + 1))
    assert not np.array_equal(u, P.block_bytes(rows, k, seed + 1, offset))


def test_handworked_roundings():
    for c in sr_handworked():
        grid = F.F_GRID if c["grid"] == "E2M1" else F.I_GRID
        got = F.stochastic_round_to_codebook(np.array([c["y"]]), grid, np.array([c["u"]]))[0]
        assert got == c["code"], c


def _paper_round(v):
    """App. D: round(q + eps - 1/2) with round = nearest, ties to even."""
    return np.round(v)


def _signed_quotients(bits, q):
    """fl32(x / s8) with the sign of X, for the chosen branch of each block."""
    rows, k = bits.shape
    x = (Q.bf16_to_f32(bits) / q.s32).astype(np.float32)
    s8 = np.repeat(F.e4m3_decode(q.scales & 0x7F).astype(np.float32), 16, axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        y = np.where(s8 > 0, np.abs(x) / s8, np.float32(0)).astype(np.float32)
    return np.where(bits >> 15, -y.astype(np.float64), y.astype(np.float64))


def _eps(rows, k, seed, offset):
    return (P.block_bytes(rows, k, seed, offset).astype(np.float64) + 0.5) / 256.0


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_int4_branch_is_appendix_d_formula(seed):
    bits = W.adversarial(40 + seed, 24, 128)
    q = Q.quantize(bits, mode="e1m2", rounding="stochastic", seed=seed, offset=seed * 11)
    ys = _signed_quotients(bits, q)
    eps = _eps(24, 128, seed, seed * 11)
    ref = np.clip(_paper_round(ys + eps - 0.5), -7, 7)
    nib = Q.unpack_nibbles(q.codes)
    assert np.array_equal(nib & 7, np.abs(ref).astype(np.uint8))
    assert np.array_equal(nib >> 3, (bits >> 15).astype(np.uint8))


@pytest.mark.parametrize("seed", [4, 5, 6])
def test_e2m1_branch_is_formula_on_uniform_pieces(seed):
    bits = W.adversarial(50 + seed, 24, 128)
    q = Q.quantize(bits, mode="e2m1", rounding="stochastic", seed=seed)
    ys = _signed_quotients(bits, q)
    eps = _eps(24, 128, seed, 0)
    a = np.abs(ys)
    step = np.where(a < 2, 0.5, np.where(a < 4, 1.0, 2.0))
    val = step * _paper_round(ys / step + eps - 0.5)
    val = np.clip(val, -6, 6)
    code = np.searchsorted(F.F_GRID, np.abs(val))
    assert np.array_equal(F.F_GRID[code], np.abs(val))
    nib = Q.unpack_nibbles(q.codes)
    assert np.array_equal(nib & 7, code.astype(np.uint8))


@pytest.mark.parametrize("mode", ["select", "e2m1", "e1m2"])
def test_matches_bruteforce(mode):
    for trial in range(3):
        bits = W.adversarial(200 + trial, 5, 64)
        seed, offset = 77 + trial, trial
        q = Q.quantize(bits, mode=mode, rounding="stochastic", seed=seed, offset=offset)
        codes, scales, _ = E.quantize(bits, mode=mode, draws=P.block_bytes(5, 64, seed, offset))
        assert np.array_equal(q.codes, np.array(codes, np.uint8))
        assert np.array_equal(q.scales, np.array(scales, np.uint8))


def test_ties_against_bruteforce():
    """Quotients a draw places exactly on a rounding midpoint, both grids."""
    rng = np.random.default_rng(3)
    for grid, book in ((F.F_GRID, E.E2M1), (F.I_GRID, E.E1M2X2)):
        lo = rng.integers(0, 7, 200)
        u = rng.integers(0, 256, 200)
        d = grid[lo + 1] - grid[lo]
        y = grid[lo] + d * (1.0 - (2 * u + 1) / 512.0)            # r + eps == 1
        got = F.stochastic_round_to_codebook(y, grid, u)
        from fractions import Fraction
        ref = [E.stochastic(Fraction(float(yy)), book, int(uu)) for yy, uu in zip(y, u)]
        assert list(got) == ref
        assert np.all(got % 2 == 0)


def test_unbiased_over_all_draws():
    """With y = lo + d m / 256 the mean over the 256 draws is y exactly; in
    general it is within d / 512 of y (the draws' resolution)."""
    u = np.arange(256)
    rng = np.random.default_rng(8)
    for grid in (F.F_GRID, F.I_GRID):
        for _ in range(200):
            lo = int(rng.integers(0, 7))
            d = grid[lo + 1] - grid[lo]
            m = int(rng.integers(0, 256))
            y = grid[lo] + d * m / 256.0
            codes = F.stochastic_round_to_codebook(np.full(256, y), grid, u)
            mean = grid[codes].mean()
            # m/256 with no ties except r + eps == 1 never occurs (eps has odd numerator)
            assert mean == y
            y2 = grid[lo] + d * float(rng.random())
            y2 = float(np.float32(y2))
            codes = F.stochastic_round_to_codebook(np.full(256, y2), grid, u)
            assert abs(grid[codes].mean() - y2) <= d / 512.0 + 1e-12


def test_scales_and_choice_are_round_to_nearest():
    bits = W.adversarial(9, 32, 256)
    qn = Q.quantize(bits)
    qs = Q.quantize(bits, rounding="stochastic", seed=5)
    assert np.array_equal(qn.scales, qs.scales)
    assert qn.s32 == qs.s32
    # the codes move by at most one grid step from round-to-nearest
    nn, ns = Q.unpack_nibbles(qn.codes), Q.unpack_nibbles(qs.codes)
    assert np.all(np.abs((nn & 7).astype(int) - (ns & 7).astype(int)) <= 1)
    assert np.array_equal(nn >> 3, ns >> 3)
    assert (nn != ns).any()


def test_on_grid_values_are_fixed():
    """Values already on a grid (times the block scale) keep their codes
    whatever the draws."""
    rng = np.random.default_rng(12)
    mags = rng.choice(F.F_GRID, size=(16, 64))
    mags[:, ::16] = 6.0
    x = mags * rng.choice([-1.0, 1.0], size=mags.shape)
    bits = W.f32_to_bf16_bits(x.astype(np.float32))
    qn = Q.quantize(bits, s32=1.0, mode="e2m1")
    for seed in range(4):
        qs = Q.quantize(bits, s32=1.0, mode="e2m1", rounding="stochastic", seed=seed)
        assert np.array_equal(qn.codes, qs.codes)


def test_row_index_matches_full_tensor():
    """Rows quantized on their own with their global row numbers get the
    codes they get inside the whole tensor."""
    bits = W.adversarial(31, 40, 96)
    full = Q.quantize(bits, s32=0.5, rounding="stochastic", seed=9, offset=2)
    rows = np.array([0, 7, 39])
    part = Q.quantize(bits[rows], s32=0.5, rounding="stochastic", seed=9, offset=2, row_index=rows)
    assert np.array_equal(part.codes, full.codes[rows])
