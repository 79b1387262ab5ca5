"""Algorithm 1 (MixFP4 data type quantization) and its inverse, on the CPU.

TEST INFRASTRUCTURE (oracle); see ``oracle/__init__``.

Follows, in order:
  Algorithm 1, tensor-scale step: s32 = max|X| / 2688 (2688 = 6*448 = 7*384).
  Algorithm 1, FP8-domain step:   X_FP8 = X / s32.
  Algorithm 1, E2M1 branch:       s8 = FP8_E4M3(block-max|X_FP8| / 6),
                                  quantize to E2M1, dequantize, MSE.
  Algorithm 1, E1M2 branch:       same with 7 and the E1M2 (x2, INT4) grid.
  Algorithm 1, selection:         E2M1 if Err_E2M1 < Err_E1M2, else E1M2 and T = 1.
  Sec. 3.2 / App. B.3:            T stored in bit 7 of the E4M3 block scale.
  App. B.2:                       nibble = [s | p2 p1 p0].
  App. B.1:                       blocks of V = 16 values along the reduction dim.
  App. D (optional):              stochastic rounding of the chosen branch's codes.

Readings of passages the paper leaves open (all listed in the design notes):
  * X_FP8 = fl32(X / s32) with IEEE fp32 division; s32 = fl32(amax / 2688),
    or 1.0 when the tensor is all zero; a caller may supply s32 instead.
  * FP8_E4M3 / FP4 rounding: nearest value, ties to even code, saturating.
    The FP4 argument is the fp32 quotient fl32(|x| / s8); rounding that is the
    same as rounding the exact quotient (checked by ``oracle.exact``).
  * MSE compares the exact real sums of squared errors (the 1/16 cancels).
  * The nibble's sign bit is the sign bit of X, also when the code is zero.
  * Layout: element 2j in the low nibble of byte j; codes [rows, K/2],
    scales [rows, K/16], both row-major.
  * Stochastic rounding: App. D's rule on the local lattice of each grid
    (see ``formats.stochastic_round_to_codebook``), applied to the fp32
    quotient, with Philox4x32-10 draws of 8 bits per element
    (``oracle.philox``); scales and the format choice stay round-to-nearest.
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction

import numpy as np

from . import formats as F
from . import philox

BLOCK = 16
TENSOR_DIVISOR = np.float32(2688.0)     # 6 * 448 = 7 * 384 (Algorithm 1)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def tensor_scale(x_bits: np.ndarray) -> np.float32:
    """Algorithm 1 tensor-scale step: fl32(max|X| / 2688), 1.0 for an all-zero X."""
    x = bf16_to_f32(x_bits)
    amax = np.float32(np.max(np.abs(x))) if x.size else np.float32(0)
    if amax == 0:
        return np.float32(1.0)
    return np.float32(amax / TENSOR_DIVISOR)


@dataclass
class Quantized:
    codes: np.ndarray      # uint8 [rows, K/2]
    scales: np.ndarray     # uint8 [rows, K/16]
    s32: np.float32
    # diagnostics (not part of the format)
    t: np.ndarray          # uint8 [rows, K/16] format bit
    sf_code: np.ndarray    # E4M3 code of the E2M1 candidate scale
    si_code: np.ndarray    # E4M3 code of the E1M2 candidate scale
    delta: np.ndarray      # float64 Err_E2M1 - Err_E1M2 (sum form), exact


def _exact_block_sums(terms: np.ndarray):
    """Sum each row of exactly representable float64 ``terms``; also return a
    mask of rows whose fp64 sum is provably exact.

    A row is certified when all its nonzero terms are integer multiples of
    2^u (u = lowest set bit over the row) and sum(|terms|) < 2^(u+53): every
    partial sum is then an integer multiple of 2^u below 2^53 * 2^u, hence
    representable, so no addition rounds."""
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


def _fraction_sum(row) -> Fraction:
    return sum((Fraction(float(t)) for t in row), Fraction(0))


def signed_draws(u: np.ndarray, sign: np.ndarray) -> np.ndarray:
    """App. D rounds the signed quotient: q + eps - 1/2 for q < 0 is the
    magnitude |q| + (1 - eps) - 1/2 negated, so a negative element uses the
    magnitude rule with eps' = 1 - eps, i.e. draw 255 - u."""
    return np.where(sign == 1, 255 - u, u)


MODES = ("select", "e2m1", "e1m2", "four_six")
ROUNDINGS = ("nearest", "stochastic")


def _algorithm1_blocks(xb: np.ndarray, mode: str):
    """Algorithm 1 after the tensor scale, on blocks ``xb`` = |X_FP8| of shape
    [..., L] (fp32; L = 16 for the 1D format, 256 for a 16x16 tile):
    candidate scales, both grids, the exact error comparison and the choice.
    Returns the E4M3 codes of both candidate scales, both code arrays, both
    fp32 quotients, the exact Err_E2M1 - Err_E1M2 and T."""
    L = xb.shape[-1]
    bm = xb.max(axis=-1)                                    # block-max |X_FP8|

    def branch(divisor, grid):
        cand = (bm / np.float32(divisor)).astype(np.float32)
        code = F.e4m3_encode(cand.astype(np.float64))
        s8 = F.e4m3_decode(code)                            # exact float64
        s8_32 = s8.astype(np.float32)
        with np.errstate(divide="ignore", invalid="ignore"):
            y = np.where(s8_32[..., None] > 0, xb / s8_32[..., None], np.float32(0)).astype(np.float32)
        q = F.round_to_codebook(y.astype(np.float64), grid)
        d = grid[q] * s8[..., None]                          # dequantized, exact in fp64
        return code, s8, q, d, y

    cf, sf, qf, df, yf = branch(6, F.F_GRID)
    if mode == "four_six":
        # the second candidate is E2M1 with the block max mapped to 4
        ci, si, qi, di, yi = branch(4, F.F_GRID)
    else:
        ci, si, qi, di, yi = branch(7, F.I_GRID)

    # Err_E2M1 - Err_E1M2 = sum((x - Df)^2 - (x - Di)^2) = sum((Di - Df) * (2x - Df - Di)).
    # Each term is exact in fp64; the block sum is certified exact or redone
    # with rationals.
    xd = xb.astype(np.float64)
    terms = (di - df) * ((2.0 * xd - df) - di)
    delta, ok = _exact_block_sums(terms.reshape(-1, L))
    if not ok.all():
        flat_terms = terms.reshape(-1, L)
        for i in np.flatnonzero(~ok):
            exact = _fraction_sum(flat_terms[i])
            delta[i] = 0.0 if exact == 0 else (1.0 if exact > 0 else -1.0) * max(abs(float(exact)), 5e-324)
    delta = delta.reshape(bm.shape)
    t = (~(delta < 0)).astype(np.uint8)                    # E2M1 iff Err_E2M1 < Err_E1M2
    if mode == "four_six":
        t = (delta > 0).astype(np.uint8)                   # /4 only where strictly better
    elif mode != "select":
        t = np.full_like(t, 0 if mode == "e2m1" else 1)
    return cf, ci, qf, qi, yf, yi, delta, t


def quantize(x_bits: np.ndarray, s32=None, mode: str = "select", rounding: str = "nearest",
             seed: int = 0, offset: int = 0, row_index=None) -> Quantized:
    """Algorithm 1 on a bf16 tensor ``x_bits`` (uint16 [rows, K], K % 16 == 0).

    ``s32`` None computes the tensor scale (Algorithm 1); otherwise the given
    fp32 value is used as s32.  ``mode`` "select" is MixFP4 (the branch with
    the smaller error, ties to E1M2).  "e2m1" and "e1m2" take one branch of
    Algorithm 1 for every block, with everything else unchanged: the E2M1
    branch alone is NVFP4 (Sec. 2.1: block scale E4M3(max/6), E2M1 codes) and
    the E1M2 branch alone is the INT4-style format, with the same tensor-scale
    rule; T still records the branch.  "four_six" is the 4/6 candidate set
    the paper compares against (Sec. 2.3, Sec. 4.2): E2M1 under the block scale
    E4M3(max/6) or E4M3(max/4), whichever has the smaller squared error
    (ties keep /6); T is 0, so the result is plain NVFP4.

    ``rounding`` "stochastic" writes the codes of the chosen branch by the
    stochastic rounding of App. D (``formats.stochastic_round_to_codebook``)
    of the same fp32 quotient y = fl32(|x| / s8), with the draws u of
    ``philox.block_bytes(rows, K, seed, offset)`` (255 - u for an element
    whose sign bit is set).  Block scales and the format choice are those of
    round-to-nearest: the choice does not depend on the draws, so each code
    stays an unbiased estimate of y on its grid.  ``row_index`` numbers the
    rows within a larger tensor (the draws depend on the block index there)."""
    assert mode in MODES and rounding in ROUNDINGS
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    rows, k = x_bits.shape
    assert k % BLOCK == 0
    s32 = tensor_scale(x_bits) if s32 is None else np.float32(s32)
    X = bf16_to_f32(x_bits)
    x = (X / s32).astype(np.float32)                       # X_FP8, IEEE fp32 division
    nb = k // BLOCK
    xb = np.abs(x).reshape(rows, nb, BLOCK)
    cf, ci, qf, qi, yf, yi, delta, t = _algorithm1_blocks(xb, mode)

    sign = (x_bits.reshape(rows, nb, BLOCK) >> 15).astype(np.uint8)
    if rounding == "stochastic":
        u = philox.block_bytes(rows, k, seed, offset, row_index).reshape(rows, nb, BLOCK)
        u = u.astype(np.int64)
        u = signed_draws(u, sign)
        qf = F.stochastic_round_to_codebook(yf, F.F_GRID, u)
        qi = F.stochastic_round_to_codebook(yi, F.F_GRID if mode == "four_six" else F.I_GRID, u)
    mag = np.where(t[..., None] == 1, qi, qf).astype(np.uint8)
    nib = (sign << 3) | mag
    nib = nib.reshape(rows, k)
    codes = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    tbit = np.zeros_like(t) if mode == "four_six" else t
    scales = ((tbit << 7) | np.where(t == 1, ci, cf)).astype(np.uint8)
    return Quantized(codes=codes, scales=scales, s32=s32, t=t,
                     sf_code=cf.astype(np.uint8), si_code=ci.astype(np.uint8), delta=delta)


def unpack_nibbles(codes: np.ndarray) -> np.ndarray:
    """uint8 [rows, K/2] -> uint8 [rows, K] nibbles (element 2j = low nibble)."""
    codes = np.asarray(codes, dtype=np.uint8)
    rows, half = codes.shape
    nib = np.empty((rows, half * 2), dtype=np.uint8)
    nib[:, 0::2] = codes & 0x0F
    nib[:, 1::2] = codes >> 4
    return nib


def decode_unit(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """s8 * v(code, T) * sign as exact float64 (the per-element value before the
    tensor scale).  T (scale bit 7) selects the E2M1 or INT4 magnitude; the
    scale magnitude is bits 6:0 (App. B.3)."""
    nib = unpack_nibbles(codes)
    rows, k = nib.shape
    scales = np.asarray(scales, dtype=np.uint8)
    t = np.repeat((scales >> 7).astype(np.int64), BLOCK, axis=1)
    s8 = np.repeat(F.e4m3_decode(scales & 0x7F), BLOCK, axis=1)
    mag = (nib & 7).astype(np.int64)
    v = np.where(t == 1, F.I_GRID[mag], F.F_GRID[mag])
    sgn = np.where(nib & 8, -1.0, 1.0)
    return sgn * v * s8


def dequantize(codes, scales, s32=None) -> np.ndarray:
    """fl32(s32 * (s8 * v)); s8 * v is exact, so this rounds once.  ``s32`` None
    gives the FP8-domain values (scale 1.0)."""
    unit = decode_unit(codes, scales)
    s = 1.0 if s32 is None else float(np.float32(s32))
    return (unit * s).astype(np.float32)


def dequantize_exact(codes, scales, s32=None) -> np.ndarray:
    """s32 * s8 * v in float64 without the final fp32 rounding (exact: at most
    24 + 4 + 3 significant bits)."""
    unit = decode_unit(codes, scales)
    s = 1.0 if s32 is None else float(np.float32(s32))
    return unit * s


@dataclass
class Quantized2D:
    """A weight quantized in 16x16 tiles, in both K-major layouts."""
    codes: np.ndarray      # uint8 [N, K/2]   (W, blocks along K)
    scales: np.ndarray     # uint8 [N, K/16]  (each tile's byte on its 16 rows)
    codes_t: np.ndarray    # uint8 [K, N/2]   (W^T, blocks along N)
    scales_t: np.ndarray   # uint8 [K, N/16]
    s32: np.float32
    t: np.ndarray          # uint8 [N/16, K/16]
    tile_scales: np.ndarray  # uint8 [N/16, K/16] scale bytes


def _pack(nib: np.ndarray) -> np.ndarray:
    return (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)


def quantize_2d(x_bits: np.ndarray, s32=None, mode: str = "select") -> Quantized2D:
    """2D block quantization of a weight W (uint16 bf16 [N, K], N and K
    multiples of 16): Algorithm 1 with the block being a 16 x 16 tile of W
    (one block max, one pair of candidate scales, one error comparison over
    the 256 elements, one T), as the FP4 training recipe the paper follows
    does for weights (Sec. 3.2, Fig. 7; Sec. 4.3).  The tensor scale is
    Algorithm 1's.  The result is written in the 1D MixFP4 layout twice:
    for W (blocks of 16 along K, the tile's scale byte repeated on its 16
    rows) and for W^T (blocks of 16 along N), so both FPROP (A W^T) and
    DGRAD (dY W = dY (W^T)^T) read it as an ordinary operand, and the two
    dequantize to exact transposes of each other."""
    assert mode in MODES
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    n, k = x_bits.shape
    assert n % BLOCK == 0 and k % BLOCK == 0
    s32 = tensor_scale(x_bits) if s32 is None else np.float32(s32)
    x = (bf16_to_f32(x_bits) / s32).astype(np.float32)
    tn, tk = n // BLOCK, k // BLOCK
    # tiles[a, b, 16 i + j] = x[16 a + i, 16 b + j]
    tiles = np.abs(x).reshape(tn, BLOCK, tk, BLOCK).transpose(0, 2, 1, 3).reshape(tn, tk, BLOCK * BLOCK)
    cf, ci, qf, qi, _, _, _, t = _algorithm1_blocks(tiles, mode)
    mag = np.where(t[..., None] == 1, qi, qf).astype(np.uint8)
    mag = mag.reshape(tn, tk, BLOCK, BLOCK).transpose(0, 2, 1, 3).reshape(n, k)
    nib = ((x_bits >> 15).astype(np.uint8) << 3) | mag
    tbit = np.zeros_like(t) if mode == "four_six" else t
    tile_scales = ((tbit << 7) | np.where(t == 1, ci, cf)).astype(np.uint8)
    scales = np.repeat(tile_scales, BLOCK, axis=0)                       # [N, K/16]
    scales_t = np.repeat(tile_scales.T, BLOCK, axis=0)                   # [K, N/16]
    return Quantized2D(codes=_pack(nib), scales=scales, codes_t=_pack(np.ascontiguousarray(nib.T)),
                       scales_t=np.ascontiguousarray(scales_t), s32=s32, t=t,
                       tile_scales=tile_scales)
