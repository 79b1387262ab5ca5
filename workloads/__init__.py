"""Seeded synthetic workloads for the MixFP4 quantizer and GEMM.

This module only draws random tensors and rounds them to bf16. It holds none
of the MixFP4 arithmetic (no scales, codebooks, rounding to FP4 grids, error
evaluation or packing), so both the CPU oracle and the HIP path may consume
its output: they then see the same bf16 bits.

The paper evaluates on LLM weights and activations (Llama / Qwen linear
layers, Sec. 4 and Table 3) that are not available here.  The recipes below
stand in for those tensors with matching shapes and the statistics the paper
describes: heavy tails and outlier channels (Sec. 1, Sec. 2.2, Figs. 2-3),
block-wise crest-factor heterogeneity, and Hadamard feature mixing
(Sec. 2.3, RHT in Table 3).

Recipe conventions (every workload):
  * ``seed`` builds a ``numpy.random.SeedSequence``; independent streams are
    spawned from it in a fixed order, one per tensor / purpose, so a tensor's
    values do not depend on which other tensors are generated.
  * Bulk draws are split into fixed chunks of ``CHUNK`` elements, each with its
    own spawned stream, and may be filled by several threads; the result is
    independent of the thread count.
  * Values are produced in float32 (float64 for the t, Laplace and Hadamard
    steps), then rounded to bf16 with round-to-nearest-even.  Tensors are
    returned as ``uint16`` bf16 bit patterns in row-major [rows, K] layout.
  * "+-U(a,b)" means a uniformly random sign times U(a, b).
  * "p% of entries" draws round(p * n) distinct flat positions.
  * "N(0, s)" has standard deviation s.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

CHUNK = 1 << 22
_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


# ----------------------------------------------------------------------------
# bf16 helpers (bit-level conversion only)
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even); return uint16 bits.

    Inputs are finite.  Works in chunks so that 2^28-element tensors do not
    need several GB of temporaries.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    flat = a.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint16)
    step = 1 << 24
    for s in range(0, flat.size, step):
        u = flat[s:s + step].view(np.uint32)
        r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
        out[s:s + step] = r.astype(np.uint16)
    return out.reshape(a.shape)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


# ----------------------------------------------------------------------------
# chunked, thread-parallel draws
# ----------------------------------------------------------------------------
def _chunked(ss: np.random.SeedSequence, n: int, fill, dtype) -> np.ndarray:
    out = np.empty(n, dtype=dtype)
    nchunks = max(1, (n + CHUNK - 1) // CHUNK)
    children = ss.spawn(nchunks)

    def work(i):
        lo, hi = i * CHUNK, min(n, (i + 1) * CHUNK)
        rng = np.random.default_rng(children[i])
        out[lo:hi] = fill(rng, hi - lo)

    if nchunks == 1:
        work(0)
    else:
        with ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(work, range(nchunks)))
    return out


def normal(ss, n, std=1.0):
    return _chunked(ss, n, lambda r, m: r.standard_normal(m, dtype=np.float32) * np.float32(std),
                    np.float32)


def student_t(ss, n, df):
    return _chunked(ss, n, lambda r, m: r.standard_t(df, m).astype(np.float32), np.float32)


def laplace(ss, n, scale=1.0):
    return _chunked(ss, n, lambda r, m: r.laplace(0.0, scale, m).astype(np.float32), np.float32)


def _replace_outliers(flat: np.ndarray, ss, frac: float, lo: float, hi: float) -> None:
    """Replace round(frac*n) distinct entries by +-U(lo, hi) (in place)."""
    rng = np.random.default_rng(ss)
    k = int(round(frac * flat.size))
    if k == 0:
        return
    pos = rng.choice(flat.size, k, replace=False)
    sign = np.where(rng.random(k) < 0.5, -1.0, 1.0)
    mag = rng.uniform(lo, hi, k)
    flat[pos] = (sign * mag).astype(np.float32)


def _scale_channels(a2d: np.ndarray, ss, count: int, factor: float) -> np.ndarray:
    """Multiply ``count`` distinct K-columns by ``factor`` (in place); return them."""
    rng = np.random.default_rng(ss)
    cols = np.sort(rng.choice(a2d.shape[1], count, replace=False))
    a2d[:, cols] *= np.float32(factor)
    return cols


def hadamard(n: int) -> np.ndarray:
    """Sylvester Hadamard matrix of order n (a power of two), entries +-1."""
    assert n > 0 and (n & (n - 1)) == 0
    h = np.ones((1, 1))
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h


def rotate_blockdiag(a2d: np.ndarray, block: int = 128) -> np.ndarray:
    """Right-multiply by blockdiag(H_block / sqrt(block)) along K (float64 math)."""
    rows, k = a2d.shape
    assert k % block == 0
    h = hadamard(block) / math.sqrt(block)
    out = np.empty((rows, k), dtype=np.float32)
    step = max(1, (1 << 22) // k)
    for r0 in range(0, rows, step):
        blk = a2d[r0:r0 + step].astype(np.float64).reshape(-1, k // block, block)
        out[r0:r0 + step] = (blk @ h).reshape(-1, k).astype(np.float32)
    return out


def block_mixture(ss, rows: int, k: int) -> np.ndarray:
    """Per 16-element block along K: with p=0.9 a flat N(0, 0.1) block, else a
    Laplace(0, 1) block with one randomly placed element multiplied by 40."""
    assert k % 16 == 0
    n = rows * k
    nb = n // 16
    s_kind, s_flat, s_lap, s_spike = ss.spawn(4)
    is_lap = _chunked(s_kind, nb, lambda r, m: r.random(m) >= 0.9, np.bool_)
    flat = normal(s_flat, n, 0.1).reshape(nb, 16)
    lap_idx = np.flatnonzero(is_lap)
    lap = laplace(s_lap, lap_idx.size * 16).reshape(-1, 16)
    spike = np.random.default_rng(s_spike).integers(0, 16, lap_idx.size)
    lap[np.arange(lap_idx.size), spike] *= np.float32(40.0)
    flat[lap_idx] = lap
    return flat.reshape(rows, k)


# ----------------------------------------------------------------------------
# the five workloads
# ----------------------------------------------------------------------------
@dataclass
class Workload:
    name: str
    seed: int
    tensors: dict = field(default_factory=dict)   # name -> uint16 [rows, K] bf16 bits
    gemms: list = field(default_factory=list)     # (a_name, w_name) pairs, C = A W^T
    notes: dict = field(default_factory=dict)


def tiny(seed: int = 0) -> Workload:
    """A[128,256] ~ N(0,1) and W[256,256] ~ N(0,0.02), each with 1% of entries
    replaced by +-U(8,20); C = A W^T [128,256]."""
    ss = np.random.SeedSequence(seed)
    sa, sao, sw, swo = ss.spawn(4)
    a = normal(sa, 128 * 256, 1.0)
    _replace_outliers(a, sao, 0.01, 8.0, 20.0)
    w = normal(sw, 256 * 256, 0.02)
    _replace_outliers(w, swo, 0.01, 8.0, 20.0)
    wl = Workload("tiny", seed)
    wl.tensors["A"] = f32_to_bf16_bits(a.reshape(128, 256))
    wl.tensors["W"] = f32_to_bf16_bits(w.reshape(256, 256))
    wl.gemms = [("A", "W")]
    return wl


def prefill_7b(seed: int = 1, tensors=("A", "W1", "W2")) -> Workload:
    """7B-class prefill linear layers.  A[2048,4096] ~ Student-t(nu=4) with 8
    fixed outlier K-channels scaled x50; W1[11008,4096] and W2[4096,4096] ~
    N(0,0.02).  C1 = A W1^T [2048,11008], C2 = A W2^T [2048,4096]."""
    ss = np.random.SeedSequence(seed)
    sa, sac, sw1, sw2 = ss.spawn(4)
    wl = Workload("prefill_7b", seed)
    if "A" in tensors:
        a = student_t(sa, 2048 * 4096, 4).reshape(2048, 4096)
        wl.notes["outlier_channels"] = _scale_channels(a, sac, 8, 50.0)
        wl.tensors["A"] = f32_to_bf16_bits(a)
    if "W1" in tensors:
        wl.tensors["W1"] = f32_to_bf16_bits(normal(sw1, 11008 * 4096, 0.02).reshape(11008, 4096))
    if "W2" in tensors:
        wl.tensors["W2"] = f32_to_bf16_bits(normal(sw2, 4096 * 4096, 0.02).reshape(4096, 4096))
    wl.gemms = [("A", "W1"), ("A", "W2")]
    return wl


def rotated(seed: int = 2, tensors=("A", "W")) -> Workload:
    """Feature-mixed operands.  A[4096,4096] ~ Student-t(nu=3) and
    W[14336,4096] ~ N(0,0.02), both right-multiplied along K by
    blockdiag(H128/sqrt(128)) before rounding to bf16 (orthogonal, so the
    product A W^T is unchanged in exact arithmetic).  C = A W^T [4096,14336]."""
    ss = np.random.SeedSequence(seed)
    sa, sw = ss.spawn(2)
    wl = Workload("rotated", seed)
    if "A" in tensors:
        a = student_t(sa, 4096 * 4096, 3).reshape(4096, 4096)
        wl.tensors["A"] = f32_to_bf16_bits(rotate_blockdiag(a))
    if "W" in tensors:
        w = normal(sw, 14336 * 4096, 0.02).reshape(14336, 4096)
        wl.tensors["W"] = f32_to_bf16_bits(rotate_blockdiag(w))
    wl.gemms = [("A", "W")]
    return wl


def decode(seed: int = 3, tensors=("A", "W")) -> Workload:
    """Memory-bound decode shape.  A[16,8192] ~ N(0,1) with 4 outlier
    K-channels x30; W[28672,8192] ~ N(0,0.02) with 0.5% of entries replaced by
    +-U(0.2,0.5), quantized offline.  C = A W^T [16,28672]."""
    ss = np.random.SeedSequence(seed)
    sa, sac, sw, swo = ss.spawn(4)
    wl = Workload("decode", seed)
    if "A" in tensors:
        a = normal(sa, 16 * 8192, 1.0).reshape(16, 8192)
        wl.notes["outlier_channels"] = _scale_channels(a, sac, 4, 30.0)
        wl.tensors["A"] = f32_to_bf16_bits(a)
    if "W" in tensors:
        w = normal(sw, 28672 * 8192, 0.02)
        _replace_outliers(w, swo, 0.005, 0.2, 0.5)
        wl.tensors["W"] = f32_to_bf16_bits(w.reshape(28672, 8192))
    wl.gemms = [("A", "W")]
    wl.notes["offline"] = ("W",)
    return wl


def large(seed: int = 4, tensors=("A", "W", "Q")) -> Workload:
    """Large prefill plus a standalone quantizer input.  A[16384,8192] is the
    block mixture (see ``block_mixture``), W[8192,8192] ~ N(0,0.02),
    C = A W^T [16384,8192].  Q[16384,16384] (2^28 elements) is a further
    block-mixture tensor used for quantize-only throughput."""
    ss = np.random.SeedSequence(seed)
    sa, sw, sq = ss.spawn(3)
    wl = Workload("large", seed)
    if "A" in tensors:
        wl.tensors["A"] = f32_to_bf16_bits(block_mixture(sa, 16384, 8192))
    if "W" in tensors:
        wl.tensors["W"] = f32_to_bf16_bits(normal(sw, 8192 * 8192, 0.02).reshape(8192, 8192))
    if "Q" in tensors:
        wl.tensors["Q"] = f32_to_bf16_bits(block_mixture(sq, 16384, 16384))
    wl.gemms = [("A", "W")]
    return wl


def train_7b(seed: int = 5, tensors=("X", "W", "dY")) -> Workload:
    """One linear layer of a 7B-class model in training (the flow of the
    paper's Fig. 7): X[2048,4096] ~ Student-t(nu=4) with 8 outlier K-channels
    x50 (as prefill_7b's A), W[11008,4096] ~ N(0,0.02), and the output
    gradient dY[2048,11008] ~ 1e-4 * Student-t(nu=3) with 16 output channels
    x20.  GEMMs: FPROP X W^T, DGRAD dY W, WGRAD dY^T X."""
    ss = np.random.SeedSequence(seed)
    sx, sxc, sw, sg, sgc = ss.spawn(5)
    wl = Workload("train_7b", seed)
    if "X" in tensors:
        x = student_t(sx, 2048 * 4096, 4).reshape(2048, 4096)
        wl.notes["outlier_channels"] = _scale_channels(x, sxc, 8, 50.0)
        wl.tensors["X"] = f32_to_bf16_bits(x)
    if "W" in tensors:
        wl.tensors["W"] = f32_to_bf16_bits(normal(sw, 11008 * 4096, 0.02).reshape(11008, 4096))
    if "dY" in tensors:
        g = (student_t(sg, 2048 * 11008, 3) * 1e-4).astype(np.float32).reshape(2048, 11008)
        wl.notes["grad_outlier_channels"] = _scale_channels(g, sgc, 16, 20.0)
        wl.tensors["dY"] = f32_to_bf16_bits(g)
    wl.gemms = [("X", "W")]
    return wl


WORKLOADS = {"tiny": tiny, "prefill_7b": prefill_7b, "rotated": rotated,
             "decode": decode, "large": large, "train_7b": train_7b}


def get(name: str, **kw) -> Workload:
    return WORKLOADS[name](**kw)


# ----------------------------------------------------------------------------
# adversarial / structured tensors for edge-case tests
# ----------------------------------------------------------------------------
def adversarial(seed: int, rows: int, k: int) -> np.ndarray:
    """A mix of block types that stress rounding and selection: all-zero
    blocks, blocks of one repeated value, integer-valued blocks, blocks with a
    single spike, tiny-magnitude blocks next to a large tensor maximum,
    negative zeros and uniform random blocks.  Returns bf16 bits [rows, k]."""
    assert k % 16 == 0
    rng = np.random.default_rng(seed)
    nb = rows * k // 16
    blocks = rng.standard_normal((nb, 16)).astype(np.float32)
    kind = rng.integers(0, 9, nb)
    blocks[kind == 0] = 0.0
    rep = kind == 1
    blocks[rep] = rng.standard_normal((rep.sum(), 1)).astype(np.float32)
    ints = kind == 2
    blocks[ints] = rng.integers(-7, 8, (ints.sum(), 16)).astype(np.float32)
    spk = np.flatnonzero(kind == 3)
    blocks[spk, rng.integers(0, 16, spk.size)] *= 300.0
    tiny_ = kind == 4
    blocks[tiny_] *= np.float32(1e-6)
    nz = kind == 5
    blocks[nz] = np.where(rng.random((nz.sum(), 16)) < 0.5, -0.0, blocks[nz] * 1e-3).astype(np.float32)
    uni = kind == 6
    blocks[uni] = rng.uniform(-1, 1, (uni.sum(), 16)).astype(np.float32)
    half = kind == 7
    blocks[half] = (rng.integers(-14, 15, (half.sum(), 16)) * 0.5).astype(np.float32)
    out = f32_to_bf16_bits(blocks.reshape(rows, k))
    # one block holds a large value so that most others sit far below the
    # tensor maximum (exercises small / subnormal E4M3 block scales)
    out.reshape(-1)[rng.integers(0, rows * k)] = f32_to_bf16_bits(np.array([30000.0], np.float32))[0]
    return out
