"""Pins for oracle.formats: codebooks and rounding against what the paper
prints (Table 1, Sec. 2.1, App. B.2, Algorithm 1) and against torch's
float8_e4m3fn as an independent library implementation of OCP E4M3."""
import numpy as np
import pytest

from oracle import formats as F
from tests._golden import table1


def test_table1_code_values():
    codes, fields, books = table1()
    assert fields[("E2M1", "bias")] == 2 ** (2 - 1) - 1
    assert fields[("E1M2", "bias")] == 2 ** (1 - 1) - 1
    for (fmt, code), value in codes.items():
        book = F.E2M1_FRACTIONS if fmt == "E2M1" else F.E1M2_RAW_FRACTIONS
        assert book[code] == value, (fmt, code)


def test_codebooks_as_printed():
    _, _, books = table1()
    assert F.E2M1_FRACTIONS == books["E2M1"]
    assert F.E1M2_RAW_FRACTIONS == books["E1M2"]
    assert F.INT4_FRACTIONS == books["INT4"]
    assert list(F.F_GRID) == [float(v) for v in books["E2M1"]]
    assert list(F.I_GRID) == [float(v) for v in books["INT4"]]


def test_scale_constants():
    _, fields, _ = table1()
    assert F.E4M3_MAX == float(fields[("E4M3", "max")])
    assert float(fields[("E4M3", "member")]) in set(F.E4M3_VALUES.tolist())
    assert fields[("TENSOR", "divisor")] == 6 * fields[("E4M3", "max")] == 7 * fields[("E4M3", "member")]
    assert F.F_MAX == 6 and F.I_MAX == 7


def test_exhaustive_16_codes_each_format():
    """All 16 nibbles (sign + 3-bit payload) decode per eq. (2) / App. B.2, and
    every E2M1 / INT4 magnitude lies in the unified E2M2 set (Sec. 3.3, App. B.5:
    E2M1 gains a zero mantissa bit; E1M2 maps into the same set)."""
    e2m2 = {F.fp_value(0, e, m, 2, 2) for e in range(4) for m in range(4)}
    for nib in range(16):
        s, p = nib >> 3, nib & 7
        f = F.fp_value(s, p >> 1, p & 1, 2, 1)
        i = 2 * F.fp_value(s, p >> 2, p & 3, 1, 2)
        assert abs(f) == F.E2M1_FRACTIONS[p] and (f < 0) == (s == 1 and p != 0)
        assert abs(i) == p                       # INT4 magnitude equals the payload
        assert abs(f) in e2m2 and abs(i) in e2m2
        # E2M1 -> E2M2: append a 0 mantissa bit (same exponent, bias 1)
        assert F.fp_value(0, p >> 1, (p & 1) << 1, 2, 2) == abs(f)


def test_e4m3_table_matches_torch():
    torch = pytest.importorskip("torch")
    codes = torch.arange(0, 127, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(ref, F.E4M3_VALUES)
    assert np.isnan(torch.tensor([0x7F], dtype=torch.uint8).view(torch.float8_e4m3fn).float().item())


def test_e4m3_rounding_matches_torch_cast():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    v = np.concatenate([
        rng.uniform(0, 448, 200000),
        np.exp(rng.uniform(np.log(1e-4), np.log(448), 200000)),
        (F.E4M3_VALUES[:-1] + F.E4M3_VALUES[1:]) / 2,          # exact ties
        np.nextafter((F.E4M3_VALUES[:-1] + F.E4M3_VALUES[1:]) / 2, 0),
        np.nextafter((F.E4M3_VALUES[:-1] + F.E4M3_VALUES[1:]) / 2, 1e9),
    ]).astype(np.float32)
    ours = F.e4m3_encode(v.astype(np.float64))
    theirs = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(ours, theirs.astype(np.int64))


def test_e4m3_saturates():
    assert F.e4m3_encode(np.array([448.0, 463.9, 464.0, 1e6]))[:].tolist() == [126] * 4


def test_round_to_codebook_ties_even_and_saturation():
    # F grid midpoints: .25 .75 1.25 1.75 2.5 3.5 5 -> even code
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    assert F.round_to_codebook(mids, F.F_GRID).tolist() == [0, 2, 2, 4, 4, 6, 6]
    assert F.round_to_codebook(np.array([k + 0.5 for k in range(7)]), F.I_GRID).tolist() == [0, 2, 2, 4, 4, 6, 6]
    assert F.round_to_codebook(np.array([6.5, 100.0]), F.F_GRID).tolist() == [7, 7]
    assert F.round_to_codebook(np.array([7.49, 9.0]), F.I_GRID).tolist() == [7, 7]
