"""Brute-force rational MixFP4 quantizer for tiny inputs.

TEST INFRASTRUCTURE (oracle); see ``oracle/__init__``.

An independent restatement of Algorithm 1 with Python ``Fraction``s that shares
no code with ``oracle.quant`` or ``oracle.formats``: it enumerates its own
codebooks from the value equation (Sec. 2.1, eq. (2)), rounds by scanning every
code for the nearest value of the *exact* rational quotient, and evaluates both
candidate errors as exact rational sums of squares (Algorithm 1's MSE).  It is
slow (about a millisecond per block) and serves as a pin on the vectorised
oracle, not as a second implementation of the GPU path.
"""
from __future__ import annotations

from fractions import Fraction


def _value(e: int, m: int, we: int, wm: int) -> Fraction:
    bias = (1 << (we - 1)) - 1
    if e:
        return Fraction(2) ** (e - bias) * Fraction((1 << wm) + m, 1 << wm)
    return Fraction(2) ** (1 - bias) * Fraction(m, 1 << wm)


# (code, magnitude) lists; E1M2 carries the x2 INT4 remap (App. B.2).
E2M1 = [(p, _value(p >> 1, p & 1, 2, 1)) for p in range(8)]
E1M2X2 = [(p, 2 * _value(p >> 2, p & 3, 1, 2)) for p in range(8)]
E4M3 = [(c, _value(c >> 3, c & 7, 4, 3)) for c in range(127)]
# E3M0 (W_E = 3, W_M = 0): the exponent-only FP4 micro-format of Sec. 2.3.
E3M0 = [(p, _value(p, 0, 3, 0)) for p in range(8)]
# candidate name -> (codebook, divisor of the block max)
BOOKS = {"e2m1": (E2M1, 6), "e1m2": (E1M2X2, 7), "e3m0": (E3M0, 16)}


def nearest(q: Fraction, book) -> tuple[int, Fraction]:
    """Scan ``book`` for the entry nearest to q >= 0; ties go to the even code;
    beyond the largest entry the largest is taken (it is then the nearest)."""
    best = None
    for code, v in book:
        d = abs(q - v)
        if best is None or d < best[0] or (d == best[0] and code % 2 == 0 and best[1] % 2 == 1):
            best = (d, code, v)
    return best[1], best[2]


def round_f32(q: Fraction) -> Fraction:
    """IEEE-754 binary32 round-to-nearest-even of a rational (finite range,
    gradual underflow).  Written from the definition: find the binade, scale to
    a 24-bit integer significand, round half to even."""
    if q == 0:
        return Fraction(0)
    sgn = -1 if q < 0 else 1
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)                       # subnormals share the minimum exponent
    scaled = a / Fraction(2) ** (e - 23)   # significand in units of the last place
    n = scaled.numerator // scaled.denominator
    rem = scaled - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return sgn * Fraction(n) * Fraction(2) ** (e - 23)


def bf16_value(bits: int) -> Fraction:
    """Exact value of a finite bf16 bit pattern (1-8-7 layout)."""
    s, e, m = bits >> 15, (bits >> 7) & 0xFF, bits & 0x7F
    assert e != 0xFF
    v = _value(e, m, 8, 7)
    return -v if s else v


def stochastic(y: Fraction, book, u: int) -> int:
    """App. D's stochastic rounding of y >= 0 between its two neighbours in
    ``book``: v = y + (eps - 1/2) * spacing with eps = (u + 1/2) / 256, then
    the nearer neighbour (ties to the even code); at or above the largest
    entry, the largest (App. D's clamp)."""
    top = max(book, key=lambda cv: cv[1])
    if y >= top[1]:
        return top[0]
    lo = max((cv for cv in book if cv[1] <= y), key=lambda cv: cv[1])
    hi = min((cv for cv in book if cv[1] > y), key=lambda cv: cv[1])
    eps = Fraction(2 * u + 1, 512)
    v = y + (eps - Fraction(1, 2)) * (hi[1] - lo[1])
    dlo, dhi = abs(v - lo[1]), abs(hi[1] - v)
    if dhi < dlo or (dhi == dlo and hi[0] % 2 == 0):
        return hi[0]
    return lo[0]


def quantize_block(xb_bits, s32: Fraction, mode: str = "select", draws=None):
    """Algorithm 1 on one 16-element block of bf16 bit patterns with a given s32.
    ``mode`` "e2m1" / "e1m2" keeps that branch regardless of the errors;
    "four_six" compares E2M1 under max/6 with E2M1 under max/4 (T = 0).
    ``draws`` (16 integers in [0, 256)) switches the chosen branch's codes to
    stochastic rounding of the fp32 quotient fl32(|x| / s8), with draw 255 - u
    for an element whose sign bit is set (App. D's signed rule); scales and
    the format choice stay those of round-to-nearest.
    Returns (scale_byte, [nibbles], err_e2m1, err_e1m2)."""
    X = [bf16_value(int(b)) for b in xb_bits]
    x = [round_f32(v / s32) for v in X]                      # X_FP8 in fp32
    bm = max(abs(v) for v in x)
    results = {}
    second = ("I", 4, E2M1) if mode == "four_six" else ("I", 7, E1M2X2)
    for name, div, book in (("F", 6, E2M1), second):
        cand = round_f32(bm / div)                           # fp32 argument of FP8_E4M3
        scode, s8 = nearest(cand, E4M3)
        codes, err = [], Fraction(0)
        for v in x:
            if s8 == 0:
                c, qv = 0, Fraction(0)
            else:
                c, qv = nearest(abs(v) / s8, book)           # exact quotient
            d = qv * s8
            err += (abs(v) - d) ** 2
            codes.append(c)
        results[name] = (scode, codes, err)
    ef, ei = results["F"][2], results["I"][2]
    t = 0 if ef < ei else 1
    if mode == "four_six":
        t = 1 if ei < ef else 0              # E2M1 under max/4 only where strictly better
    elif mode != "select":
        t = 0 if mode == "e2m1" else 1
    scode, mags, _ = results["I" if t else "F"]
    if draws is not None:
        book = E1M2X2 if (t and mode != "four_six") else E2M1
        s8 = E4M3[scode][1]
        mags = []
        for b, v, u in zip(xb_bits, x, draws):
            y = round_f32(abs(v) / s8) if s8 != 0 else Fraction(0)
            mags.append(stochastic(y, book, 255 - int(u) if int(b) >> 15 else int(u)))
    nibs = [((int(b) >> 15) << 3) | c for b, c in zip(xb_bits, mags)]
    tbit = 0 if mode == "four_six" else t
    return (tbit << 7) | scode, nibs, ef, ei


def tensor_scale(x_bits) -> Fraction:
    amax = max((abs(bf16_value(int(b))) for b in x_bits), default=Fraction(0))
    if amax == 0:
        return Fraction(1)
    return round_f32(amax / 2688)


def quantize(x_bits_2d, s32=None, mode: str = "select", draws=None):
    """Brute-force Algorithm 1 on a small [rows, K] uint16 array (``mode`` as
    in ``quantize_block``; ``draws`` None, or [rows, K] integers in [0, 256)
    for stochastic rounding).  Returns (codes bytes [rows][K/2], scale bytes
    [rows][K/16], s32 Fraction)."""
    rows = [list(map(int, r)) for r in x_bits_2d]
    flat = [b for r in rows for b in r]
    s = tensor_scale(flat) if s32 is None else Fraction(s32)
    codes, scales = [], []
    for ri, r in enumerate(rows):
        crow, srow = [], []
        for j in range(0, len(r), 16):
            dr = None if draws is None else [int(v) for v in draws[ri][j:j + 16]]
            sb, nibs, _, _ = quantize_block(r[j:j + 16], s, mode, dr)
            srow.append(sb)
            crow.extend(nibs[i] | (nibs[i + 1] << 4) for i in range(0, 16, 2))
        codes.append(crow)
        scales.append(srow)
    return codes, scales, s


def decode_value(nibble: int, scale_byte: int) -> Fraction:
    """Exact s8 * v(code, T) * sign for one element (App. B.2-B.3)."""
    t = scale_byte >> 7
    s8 = E4M3[scale_byte & 0x7F][1]
    mag = (E1M2X2 if t else E2M1)[nibble & 7][1]
    return (-1 if nibble & 8 else 1) * mag * s8


def quantize_block_variant(xb_bits, s32: Fraction, candidates):
    """One block (any length) of bf16 bit patterns under Algorithm 1 with the
    given candidate formats (names of BOOKS): each candidate's E4M3 scale of
    fl32(bm / divisor), codes scanned for the nearest value of the exact
    quotient, the exact squared error; the smallest error wins and ties go to
    the later candidate.  Returns (scale code, chosen index, [nibbles],
    [errors])."""
    X = [bf16_value(int(b)) for b in xb_bits]
    x = [round_f32(v / s32) for v in X]
    bm = max(abs(v) for v in x)
    res = []
    for name in candidates:
        book, div = BOOKS[name]
        scode, s8 = nearest(round_f32(bm / div), E4M3)
        codes, err = [], Fraction(0)
        for v in x:
            c, qv = (0, Fraction(0)) if s8 == 0 else nearest(abs(v) / s8, book)
            err += (abs(v) - qv * s8) ** 2
            codes.append(c)
        res.append((scode, codes, err))
    best = 0
    for j in range(1, len(res)):
        if res[j][2] <= res[best][2]:
            best = j
    scode, mags, _ = res[best]
    nibs = [((int(b) >> 15) << 3) | c for b, c in zip(xb_bits, mags)]
    return scode, best, nibs, [r[2] for r in res]


def quantize_variant(x_bits_2d, block: int, candidates, s32=None):
    """Brute force of ``oracle.variants.quantize_variant`` on a small array:
    (codes bytes [rows][K/2], scale bytes [rows][K/g], chosen index
    [rows][K/g], s32).  T is bit 7 of the scale byte for two candidates."""
    rows = [list(map(int, r)) for r in x_bits_2d]
    flat = [b for r in rows for b in r]
    s = tensor_scale(flat) if s32 is None else Fraction(s32)
    codes, scales, fmts = [], [], []
    for r in rows:
        crow, srow, frow = [], [], []
        for j in range(0, len(r), block):
            sc, best, nibs, _ = quantize_block_variant(r[j:j + block], s, candidates)
            t = best if len(candidates) == 2 else 0
            srow.append((t << 7) | sc)
            frow.append(best)
            crow.extend(nibs[i] | (nibs[i + 1] << 4) for i in range(0, block, 2))
        codes.append(crow)
        scales.append(srow)
        fmts.append(frow)
    return codes, scales, fmts, s

