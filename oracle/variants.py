"""Block-wise format selection over other candidate sets and block sizes.

TEST INFRASTRUCTURE (oracle); see ``oracle/__init__``.

The paper studies, besides MixFP4's pair, the selection rule of Algorithm 1
applied to other FP4 candidate sets and other block sizes:
  Sec. 2.3 (the E3M0 micro-format, power-of-two levels), Sec. 2.4 and
  Fig. 3 (candidate sets {E2M1}, {E2M1, E1M2}, {E2M1, E1M2, E3M0});
  Table 5 (block sizes g = 8, 16, 32, 64 for the sets FP4-E2, +FP4-E1,
  +FP4-E3, +E1+E3).
Every step is Algorithm 1's, with the block of g consecutive K elements in
place of 16 and one branch per candidate:
  tensor scale s32 = max|X| / 2688 and X_FP8 = fl32(X / s32) (unchanged);
  per block and candidate f: s_f = FP8_E4M3(fl32(bm / Q_f)) with Q_f the
  largest magnitude of f's grid, codes by nearest-value rounding of the
  fp32 quotient fl32(|x| / s_f) (ties to the even code, saturating);
  the candidate with the smallest exact sum of squared errors wins.

Readings of what the paper leaves open (listed in the design notes):
  * E3M0 follows eq. (1)-(2) with W_E = 3, W_M = 0: bias 3, code p has
    magnitude 2^(p - 3) for p >= 1 and 0 for p = 0, so its grid is
    {0, 1/4, 1/2, 1, 2, 4, 8, 16} and Q = 16.
  * The tensor-scale divisor stays 2688 for every set (E3M0's block scale
    bm / 16 never exceeds 2688 / 16 = 168 < 448).
  * Ties in the squared error go to the later candidate in the set's order,
    which is Algorithm 1's rule for the pair (E2M1 only when strictly better
    than E1M2).
  * The chosen candidate's index is stored in bit 7 of the scale byte when
    the set has two members (T, as in MixFP4); a set of three needs two bits,
    which the E4M3 scale byte does not have, so the index is returned in a
    separate array and bit 7 is zero.
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction

import numpy as np

from . import formats as F
from .quant import bf16_to_f32, tensor_scale


def _e3m0_magnitudes() -> np.ndarray:
    return np.array([float(F.fp_value(0, p, 0, 3, 0)) for p in range(8)], dtype=np.float64)


# grid (index = 3-bit code) and the divisor Q of each candidate
GRIDS = {
    "e2m1": (F.F_GRID, 6.0),
    "e1m2": (F.I_GRID, 7.0),          # E1M2 with the x2 remap (App. B.2)
    "e3m0": (_e3m0_magnitudes(), 16.0),
}
BLOCK_SIZES = (8, 16, 32, 64)


@dataclass
class QuantizedVariant:
    codes: np.ndarray      # uint8 [rows, K/2], element 2j in the low nibble of byte j
    scales: np.ndarray     # uint8 [rows, K/g]: E4M3 code, T in bit 7 for two candidates
    fmt: np.ndarray        # uint8 [rows, K/g]: index of the chosen candidate
    s32: np.float32
    block: int
    candidates: tuple


def _two_sum(a, b):
    """a + b in fp64 and whether it is exact (Knuth's TwoSum error term)."""
    s = a + b
    bb = s - a
    err = (a - (s - bb)) + (b - bb)
    return s, err == 0


def _split(a):
    c = 134217729.0 * a                  # Veltkamp split, 2^27 + 1
    hi = c - (c - a)
    return hi, a - hi


def _two_prod(a, b):
    """a * b in fp64 and whether it is exact (Dekker's product error term)."""
    p = a * b
    ah, al = _split(a)
    bh, bl = _split(b)
    err = ((ah * bh - p) + ah * bl + al * bh) + al * bl
    return p, err == 0


def _certified_sum(terms: np.ndarray):
    """Row sums of exact fp64 terms and a mask of rows whose sum is exact:
    all nonzero terms are multiples of 2^u and sum |terms| < 2^(u + 53)."""
    s = terms.sum(axis=-1)
    nz = terms != 0
    m, e = np.frexp(terms)
    mi = np.abs(np.ldexp(m, 53)).astype(np.int64)
    low = mi & (-mi)
    lowexp = np.where(nz, e.astype(np.float64) - 53.0 + np.log2(np.maximum(low, 1).astype(np.float64)),
                      np.inf)
    u = lowexp.min(axis=-1)
    total = np.abs(terms).sum(axis=-1) * (1.0 + 2.0 ** -40)
    ok = np.isinf(u) | (total < np.ldexp(1.0, np.clip(u + 53, -1074, 1023).astype(np.int64)))
    return s, ok


def _branch(xb: np.ndarray, bm: np.ndarray, name: str):
    """One candidate's branch of Algorithm 1 on blocks xb = |X_FP8| [..., g]:
    the E4M3 code of its scale, the grid codes and the dequantized values
    (exact in fp64)."""
    grid, q_max = GRIDS[name]
    cand = (bm / np.float32(q_max)).astype(np.float32)      # fp32 quotient, then FP8_E4M3
    code = F.e4m3_encode(cand.astype(np.float64))
    s8 = F.e4m3_decode(code)
    s8_32 = s8.astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        y = np.where(s8_32[..., None] > 0, xb / s8_32[..., None], np.float32(0)).astype(np.float32)
    q = F.round_to_codebook(y.astype(np.float64), grid)
    d = grid[q] * s8[..., None]
    return code, q, d


def _delta(xd: np.ndarray, db: np.ndarray, dj: np.ndarray) -> np.ndarray:
    """Err_b - Err_j per block, exactly: sum over the block of
    (x - D_b)^2 - (x - D_j)^2 = (D_j - D_b)(2x - D_b - D_j).  Every step is
    checked to be exact in fp64 and the block sum certified; blocks that fail
    any check are summed with rationals."""
    g = xd.shape[-1]
    f1, ok1 = _two_sum(dj, -db)
    f2a, ok2 = _two_sum(2.0 * xd, -db)
    f2, ok3 = _two_sum(f2a, -dj)
    t, ok4 = _two_prod(f1, f2)
    t = t.reshape(-1, g)
    s, ok = _certified_sum(t)
    ok &= (ok1 & ok2 & ok3 & ok4).reshape(-1, g).all(axis=-1)
    if not ok.all():
        xf, bf, jf = xd.reshape(-1, g), db.reshape(-1, g), dj.reshape(-1, g)
        for i in np.flatnonzero(~ok):
            ex = sum(((Fraction(float(bj)) - Fraction(float(bb))) *
                      (2 * Fraction(float(xx)) - Fraction(float(bb)) - Fraction(float(bj)))
                      for xx, bb, bj in zip(xf[i], bf[i], jf[i])), Fraction(0))
            s[i] = 0.0 if ex == 0 else (1.0 if ex > 0 else -1.0) * max(abs(float(ex)), 5e-324)
    return s.reshape(xd.shape[:-1])


def quantize_variant(x_bits: np.ndarray, block: int = 16, candidates=("e2m1", "e1m2"),
                     s32=None) -> QuantizedVariant:
    """Algorithm 1 with blocks of ``block`` consecutive K elements and the
    given candidate formats (any non-empty subset of GRIDS, in order)."""
    candidates = tuple(candidates)
    assert candidates and all(c in GRIDS for c in candidates)
    assert len(set(candidates)) == len(candidates)
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    rows, k = x_bits.shape
    assert block > 0 and k % block == 0
    s32 = tensor_scale(x_bits) if s32 is None else np.float32(s32)
    x = (bf16_to_f32(x_bits) / s32).astype(np.float32)      # X_FP8
    nb = k // block
    xb = np.abs(x).reshape(rows, nb, block)
    bm = xb.max(axis=-1)
    branches = [_branch(xb, bm, c) for c in candidates]
    xd = xb.astype(np.float64)
    best = np.zeros((rows, nb), dtype=np.int64)
    best_d = branches[0][2]
    for j in range(1, len(candidates)):
        dj = branches[j][2]
        take = ~(_delta(xd, best_d, dj) < 0)                 # Err_j <= Err_best: the later wins ties
        best = np.where(take, j, best)
        best_d = np.where(take[..., None], dj, best_d)
    codes = np.stack([b[1] for b in branches])              # [C, rows, nb, g]
    scodes = np.stack([b[0] for b in branches])              # [C, rows, nb]
    mag = np.take_along_axis(codes, best[None, ..., None], axis=0)[0].astype(np.uint8)
    scode = np.take_along_axis(scodes, best[None], axis=0)[0].astype(np.uint8)
    sign = (x_bits.reshape(rows, nb, block) >> 15).astype(np.uint8)
    nib = ((sign << 3) | mag).reshape(rows, k)
    packed = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    tbit = best.astype(np.uint8) if len(candidates) == 2 else np.zeros_like(scode)
    scales = ((tbit << 7) | scode).astype(np.uint8)
    return QuantizedVariant(codes=packed, scales=scales, fmt=best.astype(np.uint8), s32=s32,
                            block=block, candidates=candidates)


def decode_unit(q: QuantizedVariant) -> np.ndarray:
    """s8 * v * sign per element (exact float64), before the tensor scale."""
    nib = np.empty((q.codes.shape[0], q.codes.shape[1] * 2), dtype=np.uint8)
    nib[:, 0::2] = q.codes & 0x0F
    nib[:, 1::2] = q.codes >> 4
    fmt = np.repeat(q.fmt.astype(np.int64), q.block, axis=1)
    s8 = np.repeat(F.e4m3_decode(q.scales & 0x7F), q.block, axis=1)
    mag = (nib & 7).astype(np.int64)
    v = np.zeros(nib.shape, dtype=np.float64)
    for i, c in enumerate(q.candidates):
        v = np.where(fmt == i, GRIDS[c][0][mag], v)
    return np.where(nib & 8, -1.0, 1.0) * v * s8


def dequantize(q: QuantizedVariant) -> np.ndarray:
    """fl32(s32 * (s8 * v)): one rounding, as for MixFP4."""
    return (decode_unit(q) * float(q.s32)).astype(np.float32)


def relative_sse(x_bits: np.ndarray, q: QuantizedVariant) -> float:
    """sum (X - dequantized)^2 / sum X^2 over the tensor (a statistic; fp64)."""
    X = bf16_to_f32(x_bits).astype(np.float64)
    d = decode_unit(q) * float(q.s32)
    den = float((X * X).sum())
    return float(((X - d) ** 2).sum()) / den if den else 0.0
