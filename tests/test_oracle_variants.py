"""Pins of ``oracle.variants``: Algorithm 1's selection over other candidate
sets (E2M1, E1M2, E3M0; Sec. 2.3-2.4) and block sizes g = 8, 16, 32, 64
(Table 5).

* At g = 16 with {E2M1, E1M2} it is Algorithm 1 itself: equal to
  ``oracle.quant`` bit for bit; one-format sets equal the forced modes.
* Every set and block size agrees with the rational brute force of
  ``oracle.exact`` (its own codebooks from the value equation, every code
  scanned, exact squared errors).
* E3M0 has power-of-two levels (Sec. 2.3): eight codes, zero, then
  doubling magnitudes; with eq. (1)'s bias 2^(W_E - 1) - 1 = 3 they run from
  2^-2 to 2^4.
* Closed forms: a g-block whose second half is zero quantizes as the g/2
  block of its first half; a block on the E3M0 grid is selected exactly;
  exact ties go to the later candidate.
* Planted mistakes in the oracle are caught.
"""
from fractions import Fraction

import numpy as np
import pytest

import workloads as W
from oracle import exact as E
from oracle import quant as Q
from oracle import variants as V
from workloads import f32_to_bf16_bits

SETS = [("e2m1", "e1m2"), ("e2m1", "e3m0"), ("e2m1", "e1m2", "e3m0"), ("e3m0",), ("e1m2", "e3m0")]


def _mixed(seed, rows, k):
    rng = np.random.default_rng(seed)
    x = rng.standard_t(3, (rows, k)).astype(np.float32)
    x[0, : min(k, 32)] = -0.0
    x[1, : min(k, 16)] = np.arange(min(k, 16)) * 0.25
    if rows > 2:
        x[2] = 2.0 ** rng.integers(-6, 5, k) * rng.choice([-1, 1], k)     # powers of two
    if rows > 3:
        x[3] = rng.integers(-7, 8, k)
    return f32_to_bf16_bits(x)


def _brute_equal(bits, g, cands, s32=None):
    q = V.quantize_variant(bits, g, cands, s32)
    codes, scales, fmts, s = E.quantize_variant(bits, g, cands, s32)
    return (np.array_equal(q.codes, np.array(codes, np.uint8))
            and np.array_equal(q.scales, np.array(scales, np.uint8))
            and np.array_equal(q.fmt, np.array(fmts, np.uint8))
            and Fraction(float(q.s32)) == s)


def test_e3m0_power_of_two_levels():
    grid = V.GRIDS["e3m0"][0]
    assert grid.size == 8 and grid[0] == 0
    assert all(grid[i + 1] == 2 * grid[i] for i in range(1, 7))
    assert grid[1] == 0.25 and grid[-1] == 16 and V.GRIDS["e3m0"][1] == 16
    assert [float(v) for _, v in E.E3M0] == list(grid)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_pair_at_16_is_algorithm1(seed):
    for bits in (_mixed(seed, 8, 128), W.adversarial(seed, 6, 96)):
        q = V.quantize_variant(bits, 16, ("e2m1", "e1m2"))
        r = Q.quantize(bits)
        assert np.array_equal(q.codes, r.codes) and np.array_equal(q.scales, r.scales)
        assert q.s32 == r.s32
        assert np.array_equal(q.fmt, r.t)


def test_one_format_sets_are_the_forced_modes():
    bits = _mixed(5, 6, 64)
    for name, mode in (("e2m1", "e2m1"), ("e1m2", "e1m2")):
        q = V.quantize_variant(bits, 16, (name,))
        r = Q.quantize(bits, mode=mode)
        assert np.array_equal(q.codes, r.codes)
        assert np.array_equal(q.scales & 0x7F, r.scales & 0x7F)
        assert not (q.scales & 0x80).any() and not q.fmt.any()


@pytest.mark.parametrize("g", V.BLOCK_SIZES)
@pytest.mark.parametrize("cands", SETS)
def test_brute_force_agreement(g, cands):
    assert _brute_equal(_mixed(g, 5, 128), g, cands)
    assert _brute_equal(W.adversarial(g + 7, 3, 128), g, cands)
    assert _brute_equal(_mixed(g + 1, 4, 64), g, cands, s32=1.0)


@pytest.mark.parametrize("g", [16, 32, 64])
@pytest.mark.parametrize("cands", SETS)
def test_zero_half_reduces_block_size(g, cands):
    """Zeros round to code 0 with zero error under every candidate and leave
    the block max unchanged, so [B, 0] at block size g is B at g / 2."""
    rng = np.random.default_rng(g)
    half = rng.standard_t(4, (6, 4, g // 2)).astype(np.float32)
    full = np.concatenate([half, np.zeros_like(half)], axis=-1).reshape(6, 4 * g)
    bits_half = f32_to_bf16_bits(half.reshape(6, 2 * g))
    bits_full = f32_to_bf16_bits(full)
    s32 = Q.tensor_scale(bits_full)
    a = V.quantize_variant(bits_full, g, cands, s32)
    b = V.quantize_variant(bits_half, g // 2, cands, s32)
    assert np.array_equal(a.scales, b.scales) and np.array_equal(a.fmt, b.fmt)
    ca = a.codes.reshape(6, 4, g // 2)
    assert np.array_equal(ca[:, :, : g // 4].reshape(6, -1), b.codes)
    assert not ca[:, :, g // 4:].any()


def test_e3m0_grid_block_is_selected_exactly():
    """Values s * 2^j (s an E4M3 value, bm = 16 s): E3M0's scale is s and its
    error zero; E2M1's scale E4M3(16 s / 6) cannot reach 1/4 s and 16 s both."""
    rng = np.random.default_rng(3)
    s = 0.375                                               # E4M3 (1.5 * 2^-2)
    lv = 2.0 ** rng.integers(-2, 5, (4, 32))
    lv[:, 0] = 16.0
    x = (s * lv * rng.choice([-1.0, 1.0], lv.shape)).astype(np.float32)
    bits = f32_to_bf16_bits(x)
    q = V.quantize_variant(bits, 32, ("e2m1", "e3m0"), s32=1.0)
    assert (q.fmt == 1).all() and (q.scales >> 7 == 1).all()
    assert np.array_equal(V.dequantize(q), x)


def test_ties_go_to_the_later_candidate():
    # 48 / 6 = 8 and 48 / 16 = 3 are E4M3 values: E2M1 and E3M0 both exact
    x = np.zeros((2, 16), np.float32)
    x[0, 0] = 48.0
    bits = f32_to_bf16_bits(x)                              # row 1: all zero, a tie too
    for cands, want in ((("e2m1", "e3m0"), 1), (("e3m0", "e2m1"), 1),
                        (("e2m1", "e1m2", "e3m0"), 2)):
        q = V.quantize_variant(bits, 16, cands, s32=1.0)
        assert (q.fmt == want).all(), cands
        assert _brute_equal(bits, 16, cands, s32=1.0)
    q = V.quantize_variant(bits, 16, ("e3m0", "e2m1"), s32=1.0)
    assert V.dequantize(q)[0, 0] == 48.0


def test_dequantize_round_trip_on_grid():
    """Dequantized values re-quantize to themselves (same codes and scales)
    when the tensor scale is kept."""
    for g in V.BLOCK_SIZES:
        for cands in SETS:
            bits = _mixed(g * 3, 4, 128)
            q = V.quantize_variant(bits, g, cands)
            d = V.dequantize(q)
            assert np.isfinite(d).all()
            err = V.relative_sse(bits, q)
            assert 0 <= err < 0.05


# -- planted mistakes -------------------------------------------------------------

def _pins_pass():
    try:
        test_e3m0_power_of_two_levels()
        for g in (8, 32):
            for cands in (("e2m1", "e3m0"), ("e2m1", "e1m2", "e3m0")):
                if not _brute_equal(_mixed(g, 5, 128), g, cands):
                    return False
        test_ties_go_to_the_later_candidate()
        test_zero_half_reduces_block_size(32, ("e2m1", "e3m0"))
    except AssertionError:
        return False
    return True


def test_unmutated_variant_pins_pass():
    assert _pins_pass()


def test_catches_e3m0_bias_four(monkeypatch):
    grid, q = V.GRIDS["e3m0"]
    monkeypatch.setitem(V.GRIDS, "e3m0", (grid / 2, 8.0))
    assert not _pins_pass()


def test_catches_ties_to_the_earlier_candidate(monkeypatch):
    orig = V._delta
    monkeypatch.setattr(V, "_delta", lambda x, b, j: np.where(orig(x, b, j) == 0, -1.0, orig(x, b, j)))
    assert not _pins_pass()


def test_catches_e3m0_divisor_eight(monkeypatch):
    grid, q = V.GRIDS["e3m0"]
    monkeypatch.setitem(V.GRIDS, "e3m0", (grid, 8.0))
    assert not _pins_pass()


def test_catches_max_over_sixteen_elements(monkeypatch):
    """Block max taken over fixed 16-element groups instead of the g-block."""
    orig = V._branch

    def branch16(xb, bm, name):
        g = xb.shape[-1]
        if g > 16:
            bm = xb.reshape(*xb.shape[:-1], g // 16, 16).max(axis=-1)[..., 0]
        return orig(xb, bm, name)

    monkeypatch.setattr(V, "_branch", branch16)
    assert not _pins_pass()
