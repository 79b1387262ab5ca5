"""Number formats used by MixFP4, built from the paper's value equation.

TEST INFRASTRUCTURE (oracle); see ``oracle/__init__``.

* Sec. 2.1, eq. (1)-(2): a value with sign S, exponent field E (W_E bits) and
  mantissa field M (W_M bits) is (-1)^S 2^(E-B) (1 + M/2^W_M) for E >= 1 and
  (-1)^S 2^(1-B) M/2^W_M for E = 0, with bias B = 2^(W_E-1) - 1.
* Sec. 3.1, Table 1 and App. B.2: the FP4 payload is [s | p2 p1 p0].  E2M1
  reads e = p2p1, m = p0 (bias 1); E1M2 reads e = p2, m = p1p0 (bias 0).  No
  Inf/NaN codes.  E1M2 magnitudes are remapped by a fixed x2 to the INT4
  lattice {0..7} (Sec. 3.1, App. B.2 "integer-like codebook mapping").
* Algorithm 1 (comment on the tensor scale): 448 and 384 lie in the E4M3
  range; 448 is the OCP E4M3FN maximum (bias 7, no Inf, code 0x7F is NaN).
* App. B.3: the block scale is stored as an unsigned E4M3 magnitude in bits
  6:0; bit 7 carries the format type T.

Rounding (the paper does not state it; see the readings in the design notes):
round to the nearest codebook value, ties to the code with an even least
significant bit, saturating at the largest finite value.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np


def fp_value(s: int, e: int, m: int, we: int, wm: int) -> Fraction:
    """Eq. (2) with bias from eq. (1), as an exact rational."""
    bias = 2 ** (we - 1) - 1
    if e == 0:
        mag = Fraction(2) ** (1 - bias) * Fraction(m, 2 ** wm)
    else:
        mag = Fraction(2) ** (e - bias) * (1 + Fraction(m, 2 ** wm))
    return -mag if s else mag


def _fp4_magnitudes(we: int, wm: int) -> list[Fraction]:
    """Magnitudes of the eight non-negative codes p2p1p0 = 0..7 (App. B.2)."""
    out = []
    for p in range(8):
        e, m = p >> wm, p & ((1 << wm) - 1)
        out.append(fp_value(0, e, m, we, wm))
    return out


# E2M1: {0, .5, 1, 1.5, 2, 3, 4, 6}; code = index.
E2M1_FRACTIONS = _fp4_magnitudes(2, 1)
# E1M2 raw magnitudes {0, .5, ..., 3.5} and the x2 remap to {0..7}.
E1M2_RAW_FRACTIONS = _fp4_magnitudes(1, 2)
INT4_FRACTIONS = [2 * v for v in E1M2_RAW_FRACTIONS]

# Grids the quantizer rounds onto, in Algorithm 1's "FP8 domain" units:
# F = E2M1 (max 6), I = E1M2 x2 (max 7).
F_GRID = np.array([float(v) for v in E2M1_FRACTIONS], dtype=np.float64)
I_GRID = np.array([float(v) for v in INT4_FRACTIONS], dtype=np.float64)
F_MAX = 6.0
I_MAX = 7.0


def _e4m3_values() -> np.ndarray:
    vals = []
    for code in range(0x7F):            # 0x7F (E=15, M=7) is NaN in E4M3FN
        e, m = code >> 3, code & 7
        vals.append(float(fp_value(0, e, m, 4, 3)))
    return np.array(vals, dtype=np.float64)


# Non-negative finite E4M3FN values; index = 7-bit magnitude code.
E4M3_VALUES = _e4m3_values()
E4M3_MAX = float(E4M3_VALUES[-1])        # 448


def round_to_codebook(y: np.ndarray, values: np.ndarray) -> np.ndarray:
    """Index of the nearest entry of ``values`` (ascending, index = code) to
    each y >= 0.  Ties go to the even index; y above the last entry saturates
    to the last index.  ``y`` is float64 holding exactly representable inputs
    (fp32 values), so the distance comparisons below are exact."""
    y = np.asarray(y, dtype=np.float64)
    n = values.size
    hi = np.searchsorted(values, y, side="left")          # values[hi-1] < y <= values[hi]
    hi_c = np.minimum(hi, n - 1)
    lo_c = np.maximum(hi - 1, 0)
    d_lo = y - values[lo_c]
    d_hi = values[hi_c] - y
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi_c % 2 == 0))
    idx = np.where(pick_hi, hi_c, lo_c)
    idx = np.where(hi >= n, n - 1, idx)                    # saturate above the max
    idx = np.where(y <= values[0], 0, idx)
    return idx.astype(np.int64)


def e4m3_encode(v: np.ndarray) -> np.ndarray:
    """FP8_E4M3(v) of Algorithm 1 for v >= 0: the 7-bit magnitude code of the
    nearest E4M3FN value (ties to even code, saturate at 448)."""
    return round_to_codebook(v, E4M3_VALUES)


def e4m3_decode(code: np.ndarray) -> np.ndarray:
    """Value of a 7-bit E4M3 magnitude code (App. B.3 forces bit 7 to zero)."""
    return E4M3_VALUES[np.asarray(code, dtype=np.int64) & 0x7F]


def stochastic_round_to_codebook(y: np.ndarray, values: np.ndarray, u: np.ndarray) -> np.ndarray:
    """Stochastic rounding (App. D) of magnitudes y >= 0 onto ``values``
    (ascending, index = code) with draws u in [0, 256).

    App. D rounds the integer grid as round(q + eps - 1/2) with eps uniform on
    (0, 1), so q lands on one of its two neighbours with probability falling
    linearly with the distance.  Here, for y between neighbours lo <= y < hi
    (spacing d = hi - lo), that rule is applied on the local lattice:
    y + (eps - 1/2) d rounded to the nearer of lo and hi, ties to the even
    code, with eps = (u + 1/2) / 256.  y at or above the last value gives the
    last code (the clamp of App. D).  The caller passes u already mirrored
    for negative elements (255 - u), which makes the magnitude rule equal to
    App. D's signed one.

    The comparison z = 512 (y - lo) + (2u + 1) d against 512 d is exact in
    float64 wherever it can come out either way (y is an fp32 value)."""
    y = np.asarray(y, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    n = values.size
    lo = np.searchsorted(values, y, side="right") - 1      # values[lo] <= y < values[lo+1]
    lo = np.clip(lo, 0, n - 2)
    d = values[lo + 1] - values[lo]
    z = 512.0 * (y - values[lo]) + (2.0 * u + 1.0) * d
    full = 512.0 * d
    hi_even = (lo + 1) % 2 == 0
    idx = np.where((z > full) | ((z == full) & hi_even), lo + 1, lo)
    idx = np.where(y >= values[-1], n - 1, idx)
    return idx.astype(np.int64)
