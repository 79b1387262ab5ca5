"""GPU parity of the two-pass GEMM (mixfp4_gemm_ws with a workspace: both
operands decoded once to exact fp16 values in a blocked layout, then an fp16
GEMM) against the oracle's fp64 GEMM of the exactly dequantized operands:
|C - C_ref| <= 1e-5 * sum|a*w| + 1e-6 element-wise, as for mixfp4_gemm."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gemm as G
from oracle import quant as Q
from tests._gpu import dev_f32, dev_u8, gpu_quantize, host, log

pytestmark = pytest.mark.gpu


def _dev(q):
    return (dev_u8(q.codes), dev_u8(q.scales), dev_f32(q.s32))


def _ws(m, n, k, fill=None):
    import paper_2605_31035_amd as M
    size = M.mixfp4_gemm_workspace_size(m, n, k)
    ws = torch.empty(max(size, 1), dtype=torch.uint8, device="cuda")
    if fill is not None:
        ws.fill_(fill)
    return ws, size


def _check(c, qa, qw, rows=None, cols=None):
    if rows is not None:
        qa = Q.Quantized(codes=qa.codes[rows], scales=qa.scales[rows], s32=qa.s32, t=None,
                         sf_code=None, si_code=None, delta=None)
        qw = Q.Quantized(codes=qw.codes[cols], scales=qw.scales[cols], s32=qw.s32, t=None,
                         sf_code=None, si_code=None, delta=None)
        c = c[np.ix_(rows, cols)]
    a_hat, w_hat = G.operands(qa, qw)
    c_ref, bound = G.gemm(a_hat, w_hat)
    ok, worst = G.within_tolerance(c, c_ref, bound)
    assert ok.all(), f"{(~ok).sum()} elements out of tolerance, worst ratio {worst}"
    return worst


def test_workspace_size_formula():
    import paper_2605_31035_amd as M
    assert M.mixfp4_gemm_workspace_size(16384, 8192, 8192) == (16384 + 8192) * 8192 * 2
    assert M.mixfp4_gemm_workspace_size(300, 1000, 288) == (512 + 1024) * 288 * 2
    assert M.mixfp4_gemm_workspace_size(16, 4096, 4096) == 0      # decode shape: fused kernel
    assert M.mixfp4_gemm_workspace_size(64, 64, 48) == 0          # k % 32 != 0
    assert M.mixfp4_gemm_workspace_size(0, 64, 64) == 0


def test_integer_operands_exact():
    import paper_2605_31035_amd as M
    rng = np.random.default_rng(21)
    a = rng.integers(-7, 8, (70, 96)).astype(np.float32)
    w = rng.integers(-7, 8, (45, 96)).astype(np.float32)
    a.reshape(-1, 16)[:, 0] = 7
    w.reshape(-1, 16)[:, 0] = 7
    qa = Q.quantize(W.f32_to_bf16_bits(a), s32=1.0)
    qw = Q.quantize(W.f32_to_bf16_bits(w), s32=1.0)
    ws, size = _ws(70, 45, 96)
    assert size > 0
    c = host(M.mixfp4_gemm(_dev(qa), _dev(qw), workspace=ws))
    np.testing.assert_array_equal(c, (a.astype(np.int64) @ w.astype(np.int64).T).astype(np.float32))


@pytest.mark.parametrize("m,n,k", [(17, 1, 32), (130, 77, 64), (257, 129, 96), (300, 1000, 288),
                                   (512, 256, 1024), (256, 512, 32), (1000, 33, 4096)])
def test_ragged_shapes(m, n, k):
    """Tiles of 256 x 256 over padded operands (rows beyond m and n decode to
    nothing and their outputs are masked), K from one 32-step up, odd step
    counts."""
    import paper_2605_31035_amd as M
    qa = Q.quantize(W.adversarial(m + 2 * k, m, k))
    qw = Q.quantize(W.adversarial(n + 5 * k, n, k))
    log(f"two-pass ragged m={m} n={n} k={k}")
    ws, size = _ws(m, n, k, fill=0xFF)     # NaN bytes: padding rows must not leak
    assert size > 0
    c = host(M.mixfp4_gemm(_dev(qa), _dev(qw), workspace=ws))
    _check(c, qa, qw)


@pytest.mark.parametrize("m,n,k", [(4100, 4100, 512), (2048, 11008, 4096)])
def test_many_tiles(m, n, k):
    """More 256 x 256 tiles than CUs through the XCD-grouped order; checked in
    full (first shape) or on a sampled grid, and twice for bit-identical
    results with a differently filled workspace."""
    import paper_2605_31035_amd as M
    qa = Q.quantize(W.adversarial(m + 7, m, k))
    qw = Q.quantize(W.adversarial(n + 3, n, k))
    log(f"two-pass many tiles m={m} n={n} k={k}")
    a, w = _dev(qa), _dev(qw)
    ws1, _ = _ws(m, n, k, fill=0x00)
    ws2, _ = _ws(m, n, k, fill=0x7C)
    c1 = M.mixfp4_gemm(a, w, workspace=ws1)
    c2 = M.mixfp4_gemm(a, w, workspace=ws2)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)
    c = host(c1)
    if m * n <= 4100 * 4100:
        _check(c, qa, qw)
    else:
        rng = np.random.default_rng(m)
        rows = np.unique(np.concatenate([[0, m - 1], rng.integers(0, m, 48)]))
        cols = np.unique(np.concatenate([[0, n - 1], rng.integers(0, n, 64)]))
        _check(c, qa, qw, rows=rows, cols=cols)


@pytest.mark.parametrize("m,n,k,n1", [(2048, 11008, 4096, 8192), (4100, 4100, 512, 3840),
                                      (4096, 14336, 1024, 12288)])
def test_short_last_round_bit_identical(m, n, k, n1):
    """Shapes whose 256 x 256 tiles leave a short last round send its columns
    to 128 x 256 tiles (a second launch).  C must equal, bit for bit, the GEMMs
    of the W row slices [0, n1) and [n1, n), which each fill whole rounds or
    less than one and so run on 256 x 256 tiles only."""
    import paper_2605_31035_amd as M
    qa = Q.quantize(W.adversarial(m + 13, m, k))
    qw = Q.quantize(W.adversarial(n + 17, n, k))
    log(f"two-pass short last round m={m} n={n} k={k} split at {n1}")
    a = _dev(qa)
    wc, wsc, wts = _dev(qw)
    full = M.mixfp4_gemm(a, (wc, wsc, wts), workspace=True)
    left = M.mixfp4_gemm(a, (wc[:n1].contiguous(), wsc[:n1].contiguous(), wts), workspace=True)
    right = M.mixfp4_gemm(a, (wc[n1:].contiguous(), wsc[n1:].contiguous(), wts), workspace=True)
    torch.cuda.synchronize()
    assert torch.equal(full[:, :n1], left)
    assert torch.equal(full[:, n1:], right)
    rng = np.random.default_rng(n)
    rows = np.unique(np.concatenate([[0, m - 1], rng.integers(0, m, 40)]))
    cols = np.unique(np.concatenate([[0, n1 - 1, n1, n - 1], rng.integers(n1, n, 40)]))
    _check(host(full), qa, qw, rows=rows, cols=cols)


@pytest.mark.parametrize("m,n,k", [(2048, 4096, 1024), (300, 1000, 288), (1000, 260, 512)])
def test_small_products_on_half_tiles(m, n, k):
    """Products of at most half a round of 256 x 256 tiles run on 128 x 256
    tiles.  Rows are independent, so C must equal, bit for bit, the first m
    rows of the product with A stacked four times over, which has enough
    tiles to run on 256 x 256 tiles (2048 x 4096: two whole rounds); ragged
    shapes checked against the oracle."""
    import paper_2605_31035_amd as M
    qa = Q.quantize(W.adversarial(m + 21, m, k))
    qw = Q.quantize(W.adversarial(n + 23, n, k))
    log(f"two-pass half tiles m={m} n={n} k={k}")
    a, w = _dev(qa), _dev(qw)
    c = M.mixfp4_gemm(a, w, workspace=True)
    big = (a[0].repeat(4, 1), a[1].repeat(4, 1), a[2])
    c4 = M.mixfp4_gemm(big, w, workspace=True)
    torch.cuda.synchronize()
    assert torch.equal(c, c4[:m])
    if m * n <= 1000 * 1000:
        _check(host(c), qa, qw)
    else:
        rng = np.random.default_rng(m + n)
        rows = np.unique(np.concatenate([[0, m - 1], rng.integers(0, m, 40)]))
        cols = np.unique(np.concatenate([[0, n - 1], rng.integers(0, n, 40)]))
        _check(host(c), qa, qw, rows=rows, cols=cols)


@pytest.mark.parametrize("m,n,k,ws_bytes", [(16, 300, 4096, None), (64, 64, 48, None),
                                            (512, 512, 512, "short")])
def test_falls_back_to_fused(m, n, k, ws_bytes):
    """Where the two-pass path does not apply (decode-shape m, k % 32 != 0, a
    workspace one byte short) mixfp4_gemm_ws computes what mixfp4_gemm
    computes, bit for bit."""
    import paper_2605_31035_amd as M
    qa = Q.quantize(W.adversarial(m + 1, m, k))
    qw = Q.quantize(W.adversarial(n + 1, n, k))
    a, w = _dev(qa), _dev(qw)
    size = M.mixfp4_gemm_workspace_size(m, n, k)
    ws = torch.empty(max(1, size - 1 if ws_bytes == "short" else 4096), dtype=torch.uint8,
                     device="cuda")
    c_ws = M.mixfp4_gemm(a, w, workspace=ws)
    c = M.mixfp4_gemm(a, w)
    torch.cuda.synchronize()
    assert torch.equal(c_ws, c)


@pytest.mark.parametrize("name", ["prefill_7b", "rotated", "large"])
def test_workload_full_size(name):
    """The GEMMs of the prefill workloads in the launch configuration the
    benchmark times (GPU-quantized operands, workspace path); C checked on a
    sampled grid of rows x columns against the oracle."""
    import paper_2605_31035_amd as M
    log(f"generate {name}")
    wl = W.get(name) if name != "large" else W.get(name, tensors=("A", "W"))
    rng = np.random.default_rng(16)
    dq = {t: gpu_quantize(b) for t, b in wl.tensors.items()}
    for a_name, w_name in wl.gemms:
        a_bits, w_bits = wl.tensors[a_name], wl.tensors[w_name]
        m, n, k = a_bits.shape[0], w_bits.shape[0], a_bits.shape[1]
        log(f"{name}: two-pass gemm {a_name}{a_bits.shape} x {w_name}{w_bits.shape}^T")
        ws, size = _ws(m, n, k)
        assert size > 0
        c = host(M.mixfp4_gemm(dq[a_name], dq[w_name], workspace=ws))
        rows = np.unique(np.concatenate([[0, m - 1], rng.integers(0, m, 48)]))
        cols = np.unique(np.concatenate([[0, n - 1], rng.integers(0, n, 48)]))
        qa = Q.quantize(a_bits[rows], s32=Q.tensor_scale(a_bits))
        qw = Q.quantize(w_bits[cols], s32=Q.tensor_scale(w_bits))
        worst = _check(c[np.ix_(rows, cols)], qa, qw)
        log(f"{name} {a_name}x{w_name} ok, worst ratio {worst:.3g}")


@pytest.mark.parametrize("m,n1,n2,k", [(300, 1000, 77, 288), (2048, 4096, 1024, 4096)])
def test_decoded_operands_reused(m, n1, n2, k):
    """mixfp4_decode_operand + mixfp4_gemm_decoded, with A decoded once for
    two GEMMs, equal mixfp4_gemm_ws bit for bit (same kernels, same order)."""
    import paper_2605_31035_amd as M
    qa = Q.quantize(W.adversarial(m + 11, m, k))
    qw1 = Q.quantize(W.adversarial(n1 + 12, n1, k))
    qw2 = Q.quantize(W.adversarial(n2 + 13, n2, k))
    a, w1, w2 = _dev(qa), _dev(qw1), _dev(qw2)
    da = M.mixfp4_decode_operand(a)
    c1 = M.mixfp4_gemm_decoded(da, M.mixfp4_decode_operand(w1))
    c2 = M.mixfp4_gemm_decoded(da, M.mixfp4_decode_operand(w2))
    r1 = M.mixfp4_gemm(a, w1, workspace=True)
    r2 = M.mixfp4_gemm(a, w2, workspace=True)
    torch.cuda.synchronize()
    assert torch.equal(c1, r1) and torch.equal(c2, r2)
    if m * n2 <= 300 * 1000:
        _check(host(c2), qa, qw2)


def test_decoded_k_zero_and_empty():
    import paper_2605_31035_amd as M
    e = torch.empty((4, 0), dtype=torch.uint8, device="cuda")
    da = M.mixfp4_decode_operand((e, e, None))
    dw = M.mixfp4_decode_operand((torch.empty((3, 0), dtype=torch.uint8, device="cuda"),) * 2
                                 + (None,))
    out = torch.full((4, 3), 7.0, device="cuda")
    M.mixfp4_gemm_decoded(da, dw, out=out)
    assert torch.all(out == 0)


def _valid_rows(dec, rows, k):
    """The bytes of rows [0, rows) of a decoded operand (blocked layout: 256-row
    tiles x 32-K steps of 16 KB, 64 bytes per row and step)."""
    steps = k // 32
    b = dec.buf[: ((rows + 255) // 256) * steps * 16384].view(-1, steps, 256, 64)
    return b.permute(0, 2, 1, 3).reshape(-1, steps * 64)[:rows]


@pytest.mark.parametrize("rows,k,mode,given,pad", [
    (1, 32, "mixfp4", False, 0), (33, 96, "mixfp4", True, 0), (300, 288, "mixfp4", False, 8),
    (257, 1024, "e2m1", False, 0), (70, 512, "e1m2", True, 64), (129, 256, "four_six", False, 0),
    (2048, 4096, "mixfp4", False, 0)])
def test_quantize_decode_fused(rows, k, mode, given, pad):
    """mixfp4_quantize_decode: codes, scales and s32 equal mixfp4_quantize's
    (and the oracle's) bit for bit, the decoded operand equals
    mixfp4_decode_operand's on every real row, and a GEMM on it stays within
    the oracle's tolerance."""
    import paper_2605_31035_amd as M
    from tests._gpu import dev_bf16
    bits = W.prefill_7b().tensors["A"] if rows == 2048 else W.adversarial(rows + k, rows, k)
    log(f"quantize+decode rows={rows} k={k} mode={mode} given={given} pad={pad}")
    x = dev_bf16(bits)
    if pad:
        big = torch.zeros((rows, k + pad), dtype=torch.bfloat16, device="cuda")
        big[:, :k] = x
        x = big[:, :k]
    s32 = dev_f32(np.float32(0.37)) if given else None
    (codes, scales, ts), dec = M.mixfp4_quantize_decode(x, s32, mode=mode)
    rc, rs, rt = M.mixfp4_quantize(x, s32, mode=mode)
    torch.cuda.synchronize()
    assert torch.equal(codes, rc) and torch.equal(scales, rs) and torch.equal(ts, rt)
    if rows <= 300:
        ref = Q.quantize(bits, s32=np.float32(0.37) if given else None,
                         mode={"mixfp4": "select"}.get(mode, mode))
        np.testing.assert_array_equal(host(codes), ref.codes)
        np.testing.assert_array_equal(host(scales), ref.scales)
    dref = M.mixfp4_decode_operand((codes, scales, ts))
    assert torch.equal(_valid_rows(dec, rows, k), _valid_rows(dref, rows, k))
    n = 96
    qw = Q.quantize(W.adversarial(n + 1, n, k))
    dw = M.mixfp4_decode_operand(_dev(qw))
    c = M.mixfp4_gemm_decoded(dec, dw)
    assert torch.equal(c, M.mixfp4_gemm_decoded(dref, dw))
    qa = Q.Quantized(codes=host(codes), scales=host(scales), s32=host(ts)[0], t=None,
                     sf_code=None, si_code=None, delta=None)
    rr = np.unique(np.concatenate([[0, rows - 1], np.random.default_rng(rows).integers(0, rows, 64)]))
    _check(host(c), qa, qw, rows=rr, cols=np.arange(n))
