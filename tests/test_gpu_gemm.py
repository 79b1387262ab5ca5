"""GPU parity of mixfp4_gemm against the oracle's fp64 GEMM of the exactly
dequantized operands: |C - C_ref| <= 1e-5 * sum|a*w| + 1e-6 element-wise."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gemm as G
from oracle import quant as Q
from tests._golden import handworked_gemm
from tests._gpu import dev_bf16, dev_f32, dev_u8, gpu_quantize, host, log

pytestmark = pytest.mark.gpu


def _gemm_dev(qa, qw):
    import paper_2605_31035_amd as M
    a = (dev_u8(qa.codes), dev_u8(qa.scales), dev_f32(qa.s32))
    w = (dev_u8(qw.codes), dev_u8(qw.scales), dev_f32(qw.s32))
    c = M.mixfp4_gemm(a, w)
    torch.cuda.synchronize()
    return host(c)


def _check(c, qa, qw, rows=None, cols=None):
    if rows is not None:
        qa = _subset(qa, rows)
        qw = _subset(qw, cols)
        c = c[np.ix_(rows, cols)]
    a_hat, w_hat = G.operands(qa, qw)
    c_ref, bound = G.gemm(a_hat, w_hat)
    ok, worst = G.within_tolerance(c, c_ref, bound)
    assert ok.all(), f"{(~ok).sum()} elements out of tolerance, worst ratio {worst}"
    return worst


def _subset(q, rows):
    return Q.Quantized(codes=q.codes[rows], scales=q.scales[rows], s32=q.s32, t=None,
                       sf_code=None, si_code=None, delta=None)


def test_handworked_dot():
    g = handworked_gemm()
    bits = W.f32_to_bf16_bits(np.array([g["a"], g["w"]], np.float32))
    qa, qw = Q.quantize(bits[:1], s32=1.0), Q.quantize(bits[1:], s32=1.0)
    c = _gemm_dev(qa, qw)
    assert c[0, 0] == g["c"][0]


def test_integer_operands_exact():
    rng = np.random.default_rng(12)
    a = rng.integers(-7, 8, (70, 96)).astype(np.float32)
    w = rng.integers(-7, 8, (45, 96)).astype(np.float32)
    a.reshape(-1, 16)[:, 0] = 7
    w.reshape(-1, 16)[:, 0] = 7
    qa = Q.quantize(W.f32_to_bf16_bits(a), s32=1.0)
    qw = Q.quantize(W.f32_to_bf16_bits(w), s32=1.0)
    c = _gemm_dev(qa, qw)
    np.testing.assert_array_equal(c, (a.astype(np.int64) @ w.astype(np.int64).T).astype(np.float32))


@pytest.mark.parametrize("m,n,k", [(1, 1, 16), (130, 77, 48), (257, 129, 80), (16, 300, 4096),
                                   (128, 128, 32), (33, 1000, 272), (512, 256, 1024)])
def test_ragged_shapes(m, n, k):
    a = W.adversarial(m + k, m, k)
    w = W.adversarial(n + 3 * k, n, k)
    qa, qw = Q.quantize(a), Q.quantize(w)
    log(f"gemm ragged m={m} n={n} k={k}")
    _check(_gemm_dev(qa, qw), qa, qw)


@pytest.mark.parametrize("m,n,k", [(1, 1, 512), (5, 127, 1024), (16, 129, 512), (9, 1000, 2048),
                                   (16, 256, 8192), (3, 300, 1536), (16, 6150, 1024),
                                   (2, 7000, 1536), (16, 10250, 2048), (7, 10256, 512),
                                   (16, 12300, 1024), (1, 33, 256), (16, 500, 768),
                                   (4, 1300, 1280), (16, 1100, 11008), (13, 9000, 2816),
                                   (16, 1000, 64), (5, 3000, 320), (16, 4096, 4160),
                                   (1, 700, 2880), (13, 2000, 192), (7, 1500, 704)])
def test_decode_shapes(m, n, k):
    """m <= 16 with k % 64 == 0 takes the decode-shape kernel: K split over
    4 waves in equal shares (k % 1024 == 0) or in shares that differ by one
    256-wide step (k / 256 odd or 1 mod 4 or 3 mod 4: 1, 3, 5, 43, 11 steps;
    fewer steps than waves leave waves idle), over 2 when k / 256 is 2 mod 4;
    a tail of 64, 128 or 192 after the whole steps (0, 1, 16, 11, 0 and 2 of
    them) goes to the last wave, its lanes past the tail reading nothing;
    16, 32, 48 or 64 columns per workgroup (n up to 4096, 8192, 12288, above),
    ragged last column groups included."""
    a = W.adversarial(7 * m + k, m, k)
    w = W.adversarial(11 * n + k, n, k)
    qa, qw = Q.quantize(a), Q.quantize(w)
    log(f"gemm decode-shape m={m} n={n} k={k}")
    _check(_gemm_dev(qa, qw), qa, qw)


@pytest.mark.parametrize("m,n,k", [(4100, 4100, 512), (4100, 4100, 560)])
def test_many_tiles_ragged(m, n, k):
    """More 256x256 tiles than CUs (several waves of workgroups through the
    XCD-grouped tile order), ragged edges, fast and masked-K paths.  Checked
    in full, and twice for bit-identical results."""
    a = W.adversarial(m + 5, m, k)
    w = W.adversarial(n + 9, n, k)
    qa, qw = Q.quantize(a), Q.quantize(w)
    log(f"gemm many tiles m={m} n={n} k={k}")
    c1 = _gemm_dev(qa, qw)
    c2 = _gemm_dev(qa, qw)
    assert np.array_equal(c1, c2)
    _check(c1, qa, qw)


@pytest.mark.parametrize("m,n,k,cuts", [(2048, 11008, 512, (8192,)), (3072, 11008, 256, (8192, 8448)),
                                        (16, 12288, 1024, (4096, 10240)), (300, 9000, 512, (16, 4112))])
def test_column_slices_bit_identical(m, n, k, cuts):
    """Every output sums its K range in the same order whatever the tile
    shape, the number of launches (a short last round of 256 x 256 tiles goes
    to a second launch of 128 x 256 tiles) or the decode-shape width, so C
    restricted to a column range equals the GEMM of that range of W rows, bit
    for bit.  The full product is also checked against the oracle on sampled
    rows and columns, the cut columns included."""
    import paper_2605_31035_amd as M
    qa = Q.quantize(W.adversarial(m + 1, m, k))
    qw = Q.quantize(W.adversarial(n + 2, n, k))
    log(f"gemm column slices m={m} n={n} k={k} cuts={cuts}")
    a = (dev_u8(qa.codes), dev_u8(qa.scales), dev_f32(qa.s32))
    wc, ws, wt = dev_u8(qw.codes), dev_u8(qw.scales), dev_f32(qw.s32)
    full = M.mixfp4_gemm(a, (wc, ws, wt))
    edges = (0,) + tuple(cuts) + (n,)
    for lo, hi in zip(edges[:-1], edges[1:]):
        part = M.mixfp4_gemm(a, (wc[lo:hi], ws[lo:hi], wt))
        torch.cuda.synchronize()
        assert torch.equal(part, full[:, lo:hi]), f"columns {lo}..{hi}"
    rng = np.random.default_rng(m + n)
    rows = np.unique(np.concatenate([[0, m - 1], rng.integers(0, m, 40)]))
    cols = np.unique(np.concatenate([[0, n - 1], np.array(cuts), np.array(cuts) - 1,
                                     rng.integers(0, n, 200)]))
    _check(host(full), qa, qw, rows=rows, cols=cols)


@pytest.mark.parametrize("m,n,k", [(2000, 3100, 512), (2000, 3100, 560), (1500, 8000, 560)])
def test_mid_size_ragged(m, n, k):
    """Shapes with fewer 256x256 tiles than CUs: 2000 x 3100 takes 128x256
    tiles, 1500 x 8000 (192 tiles of 256x256, three quarters of a round)
    takes 256x256 ones; ragged in all three dimensions, fast and masked-K
    paths; checked in full."""
    a = W.adversarial(m + 11, m, k)
    w = W.adversarial(n + 13, n, k)
    qa, qw = Q.quantize(a), Q.quantize(w)
    log(f"gemm mid size m={m} n={n} k={k}")
    _check(_gemm_dev(qa, qw), qa, qw)


def test_forced_format_operands():
    """A quantized E2M1-only (NVFP4) and W E1M2-only (INT4) on the GPU: the
    GEMM decodes them through T like any MixFP4 operand."""
    import paper_2605_31035_amd as M
    a = W.adversarial(71, 300, 512)
    w = W.adversarial(72, 200, 512)
    qa = Q.quantize(a, mode="e2m1")
    qw = Q.quantize(w, mode="e1m2")
    log("gemm forced-format operands 300x200x512")
    ga = M.mixfp4_quantize(dev_bf16(a), mode="e2m1")
    gw = M.mixfp4_quantize(dev_bf16(w), mode="e1m2")
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(ga[0]), qa.codes)
    np.testing.assert_array_equal(host(gw[1]), qw.scales)
    c = M.mixfp4_gemm(ga, gw)
    torch.cuda.synchronize()
    _check(host(c), qa, qw)


def test_four_six_operands():
    """4/6 output is plain NVFP4 (T = 0): the GEMM decodes it like any
    MixFP4 operand."""
    import paper_2605_31035_amd as M
    a = W.adversarial(73, 200, 512)
    w = W.adversarial(74, 150, 512)
    qa, qw = Q.quantize(a, mode="four_six"), Q.quantize(w, mode="four_six")
    ga = M.mixfp4_quantize(dev_bf16(a), mode="four_six")
    gw = M.mixfp4_quantize(dev_bf16(w), mode="four_six")
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(ga[0]), qa.codes)
    np.testing.assert_array_equal(host(gw[1]), qw.scales)
    _check(host(M.mixfp4_gemm(ga, gw)), qa, qw)


def test_k_zero_writes_zeros():
    import paper_2605_31035_amd as M
    e = torch.empty((4, 0), dtype=torch.uint8, device="cuda")
    w = torch.empty((3, 0), dtype=torch.uint8, device="cuda")
    out = torch.full((4, 3), 7.0, device="cuda")
    M.mixfp4_gemm((e, e, None), (w, w, None), out=out)
    assert torch.all(out == 0)


def test_tiny_workload_end_to_end():
    import paper_2605_31035_amd as M
    wl = W.tiny()
    ga = gpu_quantize(wl.tensors["A"])
    gw = gpu_quantize(wl.tensors["W"])
    c = host(M.mixfp4_gemm(ga, gw))
    qa, qw = Q.quantize(wl.tensors["A"]), Q.quantize(wl.tensors["W"])
    np.testing.assert_array_equal(host(ga[0]), qa.codes)
    np.testing.assert_array_equal(host(gw[0]), qw.codes)
    log(f"tiny worst ratio {_check(c, qa, qw):.3g}")


@pytest.mark.parametrize("name", ["prefill_7b", "rotated", "decode", "large"])
def test_workload_full_size(name):
    """Full-size GEMMs of each workload from GPU-quantized operands (whose
    bit-exactness is checked in test_gpu_quantize); C checked on a sampled
    grid of rows x columns against the oracle."""
    import paper_2605_31035_amd as M
    log(f"generate {name}")
    wl = W.get(name) if name != "large" else W.get(name, tensors=("A", "W"))
    rng = np.random.default_rng(6)
    dq = {}
    for tname, bits in wl.tensors.items():
        dq[tname] = gpu_quantize(bits)
    for a_name, w_name in wl.gemms:
        a_bits, w_bits = wl.tensors[a_name], wl.tensors[w_name]
        log(f"{name}: gemm {a_name}{a_bits.shape} x {w_name}{w_bits.shape}^T")
        c = host(M.mixfp4_gemm(dq[a_name], dq[w_name]))
        rows = np.unique(np.concatenate([[0, a_bits.shape[0] - 1], rng.integers(0, a_bits.shape[0], 48)]))
        cols = np.unique(np.concatenate([[0, w_bits.shape[0] - 1], rng.integers(0, w_bits.shape[0], 48)]))
        qa = Q.quantize(a_bits[rows], s32=Q.tensor_scale(a_bits))
        qw = Q.quantize(w_bits[cols], s32=Q.tensor_scale(w_bits))
        worst = _check(c[np.ix_(rows, cols)], qa, qw)
        log(f"{name} {a_name}x{w_name} ok, worst ratio {worst:.3g}")


@pytest.mark.parametrize("m,n,k", [(16, 17000, 512), (5, 22000, 1024), (16, 28672, 512),
                                   (11, 30000, 1024), (16, 40000, 512), (9, 20000, 1472),
                                   (16, 30000, 704), (16, 28600, 512)])
def test_decode_shapes_column_splits(m, n, k):
    """Wide W on the decode-shape kernel: one range of 5 or 6 column groups
    per workgroup, 4 + 3 and 4 + 4 groups on two sets of waves at once (one
    workgroup per CU; the second set starts 64 columns into the workgroup's
    range, a sampled column), and 4 groups with several workgroups per CU
    beyond that.  W is quantized on the device (the
    quantizer's parity is tested on its own); C is checked on sampled columns,
    both ends of each workgroup's column range included, against the oracle
    quantizing those W rows with W's tensor scale; and column slices cut
    inside a workgroup's range equal the full product bit for bit."""
    import paper_2605_31035_amd as M
    a_bits = W.adversarial(m + n, m, k)
    w_bits = W.adversarial(3 * n + 1, n, k)
    log(f"gemm decode-shape split m={m} n={n} k={k}")
    qa = Q.quantize(a_bits)
    a = (dev_u8(qa.codes), dev_u8(qa.scales), dev_f32(qa.s32))
    wc, ws, wt = gpu_quantize(w_bits)
    full = M.mixfp4_gemm(a, (wc, ws, wt))
    groups = -(-n // (16 * 256))
    per = 16 * (groups if groups <= 8 else 4)
    edges = np.arange(0, n, per)
    rng = np.random.default_rng(n)
    cols = np.unique(np.concatenate([edges, np.minimum(edges + per - 1, n - 1),
                                     np.minimum(edges + 64, n - 1), [n - 1],
                                     rng.integers(0, n, 128)]))
    cols = cols[(cols >= 0) & (cols < n)]
    cols = np.unique(np.concatenate([cols[::max(1, len(cols) // 160)], [0, n - 1]]))
    qw = Q.quantize(w_bits[cols], s32=Q.tensor_scale(w_bits))
    np.testing.assert_array_equal(host(wc)[cols], qw.codes)
    worst = _check(host(full)[:, cols], qa, qw)
    lo, hi = per + 40, 3 * per + 17
    part = M.mixfp4_gemm(a, (wc[lo:hi], ws[lo:hi], wt))
    torch.cuda.synchronize()
    assert torch.equal(part, full[:, lo:hi])
    log(f"split ok, worst ratio {worst:.3g}")


@pytest.mark.parametrize("m,route", [(16, "decode"), (5, "decode"), (300, "fused"),
                                     (300, "two-pass")])
def test_every_scale_byte(m, route):
    """Hand-built operands whose 16-element blocks cycle through all 254
    finite scale bytes (every E4M3 code but the NaN one, with T = 0 and with
    T = 1) and random nibbles of both signs, through the decode-shape kernel
    (m <= 16, four blocks' scales decoded together), the fused kernel and the
    two-pass route: every block decode -- T's codebook and the E4M3 scale --
    against the oracle's dequantization, at tensor scales that are not powers
    of two."""
    import paper_2605_31035_amd as M
    rng = np.random.default_rng(40 + m)
    n, k = 64, 1024
    finite = np.array([b for b in range(256) if (b & 0x7F) != 0x7F], np.uint8)

    def operand(rows, s32):
        nb = rows * (k // 16)
        sc = np.resize(rng.permutation(finite), nb)
        rng.shuffle(sc)
        codes = rng.integers(0, 256, (rows, k // 2), dtype=np.uint8)
        return Q.Quantized(codes=codes, scales=sc.reshape(rows, k // 16), s32=np.float32(s32),
                           t=None, sf_code=None, si_code=None, delta=None)

    qa, qw = operand(m, 0.37), operand(n, 1.9)
    assert set(np.unique(np.concatenate([qa.scales.ravel(), qw.scales.ravel()]))) == set(finite)
    log(f"gemm every scale byte m={m} route={route}")
    a = (dev_u8(qa.codes), dev_u8(qa.scales), dev_f32(qa.s32))
    w = (dev_u8(qw.codes), dev_u8(qw.scales), dev_f32(qw.s32))
    c = M.mixfp4_gemm(a, w, workspace=True if route == "two-pass" else None)
    torch.cuda.synchronize()
    _check(host(c), qa, qw)
