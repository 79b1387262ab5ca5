"""Planted mistakes: each test breaks the CPU oracle in one plausible way
(monkeypatched, on the CPU only) and checks that the pins above catch it.
This guards the pins themselves: a pin set that passes a broken oracle would
not be evidence of anything."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import exact as E
from oracle import formats as F
from oracle import quant as Q
from tests._golden import handworked_blocks
from workloads import f32_to_bf16_bits


def _pins_pass() -> bool:
    """Hand-worked blocks plus brute-force agreement on a small mixed tensor."""
    cases = handworked_blocks()
    bits = f32_to_bf16_bits(np.stack([c["block"] for c in cases]))
    q = Q.quantize(bits, s32=1.0)
    for i, c in enumerate(cases):
        if q.scales[i, 0] != c["scale"] or bytes(q.codes[i]) != c["codes"]:
            return False
    rng = np.random.default_rng(99)
    x = rng.standard_t(3, (8, 64)).astype(np.float32)
    x[0, :16] = -0.0
    x[1, :16] = np.arange(16) * 0.25
    x[2, :16] = rng.integers(-7, 8, 16)
    bits = f32_to_bf16_bits(x)
    q = Q.quantize(bits)
    codes, scales, s = E.quantize(bits)
    return (np.array_equal(q.codes, np.array(codes, np.uint8))
            and np.array_equal(q.scales, np.array(scales, np.uint8))
            and Fraction(float(q.s32)) == s)


def test_unmutated_pins_pass():
    assert _pins_pass()


def test_catches_ties_to_lower_code(monkeypatch):
    orig = F.round_to_codebook

    def ties_down(y, values):
        idx = orig(y, values)
        y = np.asarray(y, np.float64)
        lo = np.maximum(idx - 1, 0)
        tie = (idx > 0) & (values[idx] - y == y - values[lo])
        return np.where(tie, lo, idx)

    monkeypatch.setattr(F, "round_to_codebook", ties_down)
    assert not _pins_pass()


def test_catches_selection_tie_to_e2m1(monkeypatch):
    orig = Q.quantize

    def mutated(x_bits, s32=None):
        q = orig(x_bits, s32)
        flip = (q.delta == 0)
        q.scales = np.where(flip, q.sf_code, q.scales).astype(np.uint8)
        return q

    monkeypatch.setattr(Q, "quantize", mutated)
    assert not _pins_pass()


def test_catches_swapped_divisors(monkeypatch):
    orig_encode = F.e4m3_encode
    calls = {"n": 0}

    def swapped(v):
        # first call is the E2M1 branch (bm/6): feed it bm/7 instead, and vice versa
        calls["n"] += 1
        factor = 6.0 / 7.0 if calls["n"] % 2 == 1 else 7.0 / 6.0
        return orig_encode(np.asarray(v, np.float64) * factor)

    monkeypatch.setattr(F, "e4m3_encode", swapped)
    assert not _pins_pass()


def test_catches_nibble_order(monkeypatch):
    orig = Q.quantize

    def mutated(x_bits, s32=None):
        q = orig(x_bits, s32)
        q.codes = ((q.codes >> 4) | (q.codes << 4)).astype(np.uint8)
        return q

    monkeypatch.setattr(Q, "quantize", mutated)
    assert not _pins_pass()


def test_catches_missing_int4_remap(monkeypatch):
    monkeypatch.setattr(F, "I_GRID", F.I_GRID / 2)
    assert not _pins_pass()


def test_catches_dropped_zero_sign(monkeypatch):
    orig = Q.quantize

    def mutated(x_bits, s32=None):
        q = orig(x_bits, s32)
        nib = Q.unpack_nibbles(q.codes)
        nib = np.where((nib & 7) == 0, 0, nib).astype(np.uint8)
        q.codes = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
        return q

    monkeypatch.setattr(Q, "quantize", mutated)
    assert not _pins_pass()


def test_catches_inverted_selection(monkeypatch):
    orig = Q._exact_block_sums

    def neg(terms):
        s, ok = orig(terms)
        return -s, ok

    monkeypatch.setattr(Q, "_exact_block_sums", neg)
    assert not _pins_pass()


def test_catches_wrong_tensor_divisor(monkeypatch):
    monkeypatch.setattr(Q, "TENSOR_DIVISOR", np.float32(2687.0))
    assert not _pins_pass()


def _forced_pins_pass() -> bool:
    """The forced-mode pins (tests/test_oracle_forced.py) as one predicate."""
    from tests import test_oracle_forced as TF
    try:
        TF.test_e2m1_mode_is_nvfp4()
        TF.test_e1m2_mode_is_int4()
        TF.test_forced_matches_bruteforce("e2m1", 0, None)
        TF.test_forced_matches_bruteforce("e1m2", 1, 0.37)
    except AssertionError:
        return False
    return True


def test_unmutated_forced_pins_pass():
    assert _forced_pins_pass()


def test_catches_forced_mode_ignored(monkeypatch):
    orig = Q.quantize
    monkeypatch.setattr(Q, "quantize", lambda x_bits, s32=None, mode="select": orig(x_bits, s32))
    assert not _forced_pins_pass()


def test_catches_forced_mode_wrong_scale(monkeypatch):
    orig = Q.quantize

    def mutated(x_bits, s32=None, mode="select"):
        q = orig(x_bits, s32, mode)
        if mode == "e1m2":      # E1M2 codes under the E2M1 branch's scale
            q.scales[:] = (q.scales & 0x80) | q.sf_code
        return q

    monkeypatch.setattr(Q, "quantize", mutated)
    assert not _forced_pins_pass()


def _sr_pins_pass() -> bool:
    """The stochastic-rounding pins (tests/test_oracle_sr.py) as one predicate."""
    from tests import test_oracle_sr as TS
    try:
        TS.test_handworked_roundings()
        TS.test_int4_branch_is_appendix_d_formula(1)
        TS.test_e2m1_branch_is_formula_on_uniform_pieces(4)
        TS.test_ties_against_bruteforce()
        TS.test_scales_and_choice_are_round_to_nearest()
    except AssertionError:
        return False
    return True


def test_unmutated_sr_pins_pass():
    assert _sr_pins_pass()


def test_catches_sr_without_half_offset(monkeypatch):
    orig = F.stochastic_round_to_codebook
    # eps = u / 256 instead of (u + 1/2) / 256: equivalent to shifting u by -1/2
    monkeypatch.setattr(F, "stochastic_round_to_codebook",
                        lambda y, values, u: orig(y, values, np.asarray(u, np.float64) - 0.5))
    assert not _sr_pins_pass()


def test_catches_sr_unmirrored_negatives(monkeypatch):
    monkeypatch.setattr(Q, "signed_draws", lambda u, sign: u)
    assert not _sr_pins_pass()


def test_catches_sr_ties_down(monkeypatch):
    orig = F.stochastic_round_to_codebook

    def ties_down(y, values, u):
        idx = orig(y, values, u)
        y = np.asarray(y, np.float64)
        u = np.asarray(u, np.float64)
        lo = np.searchsorted(values, y, side="right") - 1
        lo = np.clip(lo, 0, values.size - 2)
        d = values[lo + 1] - values[lo]
        tie = 512.0 * (y - values[lo]) + (2.0 * u + 1.0) * d == 512.0 * d
        return np.where(tie & (y < values[-1]), lo, idx)

    monkeypatch.setattr(F, "stochastic_round_to_codebook", ties_down)
    assert not _sr_pins_pass()


def _hadamard_pins_pass() -> bool:
    from tests import test_oracle_hadamard as TH
    try:
        TH.test_unit_vectors()
        TH.test_matches_rational_butterflies(32)
        TH.test_near_midpoint_elements(128)
        TH.test_signs_act_on_inputs()
        TH.test_overflow_and_zeros()
    except AssertionError:
        return False
    return True


def test_unmutated_hadamard_pins_pass():
    assert _hadamard_pins_pass()


def test_catches_hadamard_signs_on_outputs(monkeypatch):
    from oracle import hadamard as HD
    orig = HD.hadamard

    def on_outputs(x_bits, b, signs=None):
        y = orig(x_bits, b)
        if signs is None:
            return y
        flip = np.tile(np.asarray(signs) < 0, y.shape[1] // b)
        return np.where(flip[None, :] & ((y & 0x7FFF) != 0), y ^ 0x8000, y).astype(np.uint16)

    monkeypatch.setattr(HD, "hadamard", on_outputs)
    assert not _hadamard_pins_pass()


def test_catches_hadamard_double_rounding(monkeypatch):
    from oracle import hadamard as HD
    orig = HD.round_to_bf16
    # round to fp32 first, then to bf16
    monkeypatch.setattr(HD, "round_to_bf16",
                        lambda y: orig(np.asarray(y, np.float64).astype(np.float32).astype(np.float64)))
    assert not _hadamard_pins_pass()


def test_catches_hadamard_unnormalized(monkeypatch):
    from oracle import hadamard as HD
    monkeypatch.setattr(HD, "sylvester", lambda b, _o=HD.sylvester: 2 * _o(b))
    assert not _hadamard_pins_pass()


def _four_six_pins_pass() -> bool:
    from tests import test_oracle_four_six as T46
    try:
        T46.test_matches_bruteforce(2, 1.0)
        T46.test_ties_keep_six()
        T46.test_by_construction()
    except AssertionError:
        return False
    return True


def test_unmutated_four_six_pins_pass():
    assert _four_six_pins_pass()


def test_catches_four_six_ties_to_four(monkeypatch):
    orig = Q._algorithm1_blocks

    def mutated(xb, mode):
        out = list(orig(xb, mode))
        if mode == "four_six":
            out[7] = (out[6] >= 0).astype(np.uint8)
        return tuple(out)

    monkeypatch.setattr(Q, "_algorithm1_blocks", mutated)
    assert not _four_six_pins_pass()


def test_catches_four_six_wrong_divisor(monkeypatch):
    orig = Q._algorithm1_blocks

    def mutated(xb, mode):
        # 4/6 run as MixFP4 selection: INT4 codes under max/7 instead of E2M1 under max/4
        return orig(xb, "select" if mode == "four_six" else mode)

    monkeypatch.setattr(Q, "_algorithm1_blocks", mutated)
    assert not _four_six_pins_pass()


# --- dequantize (App. B.2-B.3): one rounding of s32 * s8 * v -----------------

def test_unmutated_dequantize_pins_pass():
    from tests.test_oracle_dequantize import dequantize_pins_pass
    assert dequantize_pins_pass()


def test_catches_dequantize_double_rounding(monkeypatch):
    """s32 * s8 rounded to fp32 first, then times v (two roundings)."""
    from tests.test_oracle_dequantize import dequantize_pins_pass

    def twice(codes, scales, s32=None):
        nib = Q.unpack_nibbles(codes)
        sc = np.asarray(scales, dtype=np.uint8)
        t = np.repeat((sc >> 7).astype(np.int64), Q.BLOCK, axis=1)
        s8 = np.repeat(F.e4m3_decode(sc & 0x7F), Q.BLOCK, axis=1)
        mag = (nib & 7).astype(np.int64)
        v = np.where(t == 1, F.I_GRID[mag], F.F_GRID[mag]) * np.where(nib & 8, -1.0, 1.0)
        s = np.float32(1.0 if s32 is None else s32)
        return (np.float32(s) * s8.astype(np.float32)).astype(np.float32) * v.astype(np.float32)

    monkeypatch.setattr(Q, "dequantize", twice)
    assert not dequantize_pins_pass()
