"""GPU parity of the training-GEMM operands (the FP4 training recipe of
Sec. 3.2 / Fig. 7): 2D (16x16-tile) weight quantization in both layouts,
transposed quantization (with stochastic rounding and a Hadamard rotation
along the rows), and the FPROP / DGRAD / WGRAD products built from them,
against the CPU oracle."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gemm as G
from oracle import hadamard as HD
from oracle import quant as Q
from tests._gpu import dev_bf16, dev_f32, host, log

pytestmark = pytest.mark.gpu

SEED = 0x0123456789ABCDEF


def _padded(bits, pad):
    x = dev_bf16(bits)
    if pad:
        rows, k = bits.shape
        big = torch.zeros((rows, k + pad), dtype=torch.bfloat16, device="cuda")
        big[:, :k] = x
        x = big[:, :k]
    return x


def _weight(seed, n, k):
    rng = np.random.default_rng(seed)
    w = rng.normal(0, 0.02, (n, k))
    w[rng.random((n, k)) < 0.005] *= 30
    if n >= 32 and k >= 32:
        w[:16, :16] = 0.0
        w[16:32, 16:32] = np.arange(256).reshape(16, 16) * 0.001
    return W.f32_to_bf16_bits(w.astype(np.float32))


def _grad(seed, t, n, scale=1e-3):
    rng = np.random.default_rng(seed)
    g = rng.standard_t(4, (t, n)) * scale
    g[:, rng.integers(0, n, 3)] *= 20
    return W.f32_to_bf16_bits(g.astype(np.float32))


# ---------------------------------------------------------------- 2D weights

@pytest.mark.parametrize("mode,omode", [("mixfp4", "select"), ("e2m1", "e2m1"), ("e1m2", "e1m2"),
                                        ("four_six", "four_six")])
@pytest.mark.parametrize("n,k,s32,pad", [(16, 16, None, 0), (48, 64, None, 0), (80, 48, 0.001, 0),
                                         (256, 512, None, 8), (272, 1040, 0.01, 0)])
def test_quantize_2d(mode, omode, n, k, s32, pad):
    import paper_2605_31035_amd as M
    bits = _weight(n + k, n, k)
    label = f"2d {mode} {n}x{k} s32={s32} pad={pad}"
    log(label)
    ts = None if s32 is None else dev_f32(s32)
    (c, s, s32d), (ct, st, _) = M.mixfp4_quantize_2d(_padded(bits, pad), ts, mode=mode)
    torch.cuda.synchronize()
    ref = Q.quantize_2d(bits, s32=s32, mode=omode)
    assert host(s32d)[0] == ref.s32
    np.testing.assert_array_equal(host(s), ref.scales, err_msg=label)
    np.testing.assert_array_equal(host(c), ref.codes, err_msg=label)
    np.testing.assert_array_equal(host(st), ref.scales_t, err_msg=label)
    np.testing.assert_array_equal(host(ct), ref.codes_t, err_msg=label)
    (c2, s2, _), none = M.mixfp4_quantize_2d(_padded(bits, pad), ts, mode=mode, transposed=False)
    assert none is None
    np.testing.assert_array_equal(host(c2), ref.codes)
    np.testing.assert_array_equal(host(s2), ref.scales)


def test_quantize_2d_full_size():
    """W2 of the 7B-class prefill workload (4096 x 4096), both layouts in full."""
    import paper_2605_31035_amd as M
    bits = W.get("prefill_7b", tensors=("W2",)).tensors["W2"]
    log("2d full size W2 4096x4096")
    (c, s, s32), (ct, st, _) = M.mixfp4_quantize_2d(dev_bf16(bits))
    torch.cuda.synchronize()
    ref = Q.quantize_2d(bits)
    assert host(s32)[0] == ref.s32
    np.testing.assert_array_equal(host(s), ref.scales)
    np.testing.assert_array_equal(host(c), ref.codes)
    np.testing.assert_array_equal(host(st), ref.scales_t)
    np.testing.assert_array_equal(host(ct), ref.codes_t)


def test_quantize_2d_many_super_blocks():
    """W [8448, 8192]: 66 x 64 = 4224 super-blocks of 128 x 128 elements, more
    than the 4096 workgroups of the launch, so the workgroups that take the
    last 256 rows do so in a second super-block.  Tiles are independent for a
    given s32, so the oracle quantizes three 256-row bands (first, middle,
    last) and both layouts are compared there."""
    import paper_2605_31035_amd as M
    n, k = 8448, 8192
    rng = np.random.default_rng(23)
    x = rng.standard_normal((n, k), dtype=np.float32)
    x *= np.float32(0.02)
    bits = W.f32_to_bf16_bits(x)
    del x
    s32 = np.float32(0.1 / 2688)   # a few elements saturate at 6 * 448 * s32
    log(f"2d {n}x{k} s32={s32} sampled bands")
    (c, s, _), (ct, st, _) = M.mixfp4_quantize_2d(dev_bf16(bits), dev_f32(s32))
    torch.cuda.synchronize()
    c, s, ct, st = host(c), host(s), host(ct), host(st)
    for r0 in (0, 4096, n - 256):
        ref = Q.quantize_2d(bits[r0:r0 + 256], s32=s32)
        label = f"band rows {r0}..{r0 + 256}"
        np.testing.assert_array_equal(s[r0:r0 + 256], ref.scales, err_msg=label)
        np.testing.assert_array_equal(c[r0:r0 + 256], ref.codes, err_msg=label)
        np.testing.assert_array_equal(st[:, r0 // 16:(r0 + 256) // 16], ref.scales_t, err_msg=label)
        np.testing.assert_array_equal(ct[:, r0 // 2:(r0 + 256) // 2], ref.codes_t, err_msg=label)


# ---------------------------------------------------------------- transposed quantization

def _ref_t(bits, s32, omode, rounding, seed, offset, b, signs):
    xt = np.ascontiguousarray(bits.T)
    if b:
        xt = HD.hadamard(xt, b, signs)
    return Q.quantize(xt, s32=s32, mode=omode, rounding=rounding, seed=seed, offset=offset)


@pytest.mark.parametrize("mode,omode", [("mixfp4", "select"), ("e2m1", "e2m1"),
                                        ("four_six", "four_six")])
@pytest.mark.parametrize("rounding", ["nearest", "stochastic"])
@pytest.mark.parametrize("b", [0, 16, 32, 64])
@pytest.mark.parametrize("rows,k,s32,pad", [(64, 64, None, 0), (320, 112, None, 8),
                                            (128, 80, 0.002, 0), (64, 16, None, 0)])
def test_quantize_transposed(mode, omode, rounding, b, rows, k, s32, pad):
    import paper_2605_31035_amd as M
    if b and rows % b:
        pytest.skip("rows not a multiple of the Hadamard block")
    bits = _grad(rows * 7 + k, rows, k)
    rng = np.random.default_rng(b + rows)
    signs = rng.choice([-1, 1], size=b) if b else None
    sd = None if signs is None else torch.tensor(signs.astype(np.int8), device="cuda")
    label = f"transposed {mode} {rounding} b={b} {rows}x{k} s32={s32} pad={pad}"
    log(label)
    ts = None if s32 is None else dev_f32(s32)
    c, s, s32d = M.mixfp4_quantize(_padded(bits, pad), ts, mode=mode, rounding=rounding,
                                   seed=SEED, offset=5, hadamard_block=b, hadamard_signs=sd,
                                   transpose=True)
    torch.cuda.synchronize()
    ref = _ref_t(bits, s32, omode, rounding, SEED, 5, b, signs)
    assert host(s32d)[0] == ref.s32, label
    np.testing.assert_array_equal(host(s), ref.scales, err_msg=label)
    np.testing.assert_array_equal(host(c), ref.codes, err_msg=label)


# ---------------------------------------------------------------- the three GEMMs

def _check_gemm(c, qa, qw, label):
    a_hat, w_hat = G.operands(qa, qw)
    c_ref, bound = G.gemm(a_hat, w_hat)
    ok, worst = G.within_tolerance(host(c), c_ref, bound)
    assert ok.all(), f"{label}: {(~ok).sum()} out of tolerance, worst {worst}"
    log(f"{label} worst ratio {worst:.3g}")


def test_fprop_dgrad_wgrad_small():
    """Y = X W^T, dX = dY W (W^T layout of the 2D weight), dW = dY^T X (both
    operands quantized transposed, with a 16-row rotation and stochastic
    rounding of the gradient)."""
    import paper_2605_31035_amd as M
    t, d_in, d_out = 256, 160, 192
    xb = W.adversarial(3, t, d_in)
    wb = _weight(4, d_out, d_in)
    gb = _grad(5, t, d_out)
    rng = np.random.default_rng(6)
    signs = rng.choice([-1, 1], size=16)
    sd = torch.tensor(signs.astype(np.int8), device="cuda")
    qx = M.mixfp4_quantize(dev_bf16(xb))
    qw, qwt = M.mixfp4_quantize_2d(dev_bf16(wb))
    qg = M.mixfp4_quantize(dev_bf16(gb), rounding="stochastic", seed=SEED)
    qgt = M.mixfp4_quantize(dev_bf16(gb), rounding="stochastic", seed=SEED, offset=1,
                            hadamard_block=16, hadamard_signs=sd, transpose=True)
    qxt = M.mixfp4_quantize(dev_bf16(xb), hadamard_block=16, hadamard_signs=sd, transpose=True)
    y = M.mixfp4_gemm(qx, qw)
    dx = M.mixfp4_gemm(qg, qwt)
    dw = M.mixfp4_gemm(qgt, qxt)
    torch.cuda.synchronize()
    rx = Q.quantize(xb)
    r2d = Q.quantize_2d(wb)
    rw = Q.Quantized(codes=r2d.codes, scales=r2d.scales, s32=r2d.s32, t=None, sf_code=None,
                     si_code=None, delta=None)
    rwt = Q.Quantized(codes=r2d.codes_t, scales=r2d.scales_t, s32=r2d.s32, t=None,
                      sf_code=None, si_code=None, delta=None)
    rg = Q.quantize(gb, rounding="stochastic", seed=SEED)
    rgt = _ref_t(gb, None, "select", "stochastic", SEED, 1, 16, signs)
    rxt = _ref_t(xb, None, "select", "nearest", 0, 0, 16, signs)
    for got, ref in ((qx, rx), (qg, rg), (qgt, rgt), (qxt, rxt)):
        np.testing.assert_array_equal(host(got[0]), ref.codes)
        np.testing.assert_array_equal(host(got[1]), ref.scales)
    _check_gemm(y, rx, rw, "fprop")
    _check_gemm(dx, rg, rwt, "dgrad")
    _check_gemm(dw, rgt, rxt, "wgrad")
    # DGRAD through the W^T layout equals the transpose-free route on the
    # dequantized weight: dX = dY W_hat
    w_hat = Q.dequantize_exact(r2d.codes, r2d.scales, r2d.s32)
    wt_hat = Q.dequantize_exact(r2d.codes_t, r2d.scales_t, r2d.s32)
    assert np.array_equal(w_hat.T, wt_hat)


def test_wgrad_full_size():
    """dW = dY^T X for the 7B-class layer (T = 2048 tokens, 4096 -> 11008):
    both operands quantized transposed with a 16-row random Hadamard
    rotation, the gradient with stochastic rounding; sampled rows and
    columns of dW against the oracle."""
    import paper_2605_31035_amd as M
    t, d_in, d_out = 2048, 4096, 11008
    xb = W.get("prefill_7b", tensors=("A",)).tensors["A"]
    gb = _grad(7, t, d_out)
    signs = np.random.default_rng(8).choice([-1, 1], size=16)
    sd = torch.tensor(signs.astype(np.int8), device="cuda")
    log("wgrad full size: quantize transposed")
    qgt = M.mixfp4_quantize(dev_bf16(gb), rounding="stochastic", seed=SEED, hadamard_block=16,
                            hadamard_signs=sd, transpose=True)
    qxt = M.mixfp4_quantize(dev_bf16(xb), hadamard_block=16, hadamard_signs=sd, transpose=True)
    dw = host(M.mixfp4_gemm(qgt, qxt))
    torch.cuda.synchronize()
    rng = np.random.default_rng(9)
    ro = np.unique(np.concatenate([[0, d_out - 1], rng.integers(0, d_out, 40)]))
    ri = np.unique(np.concatenate([[0, d_in - 1], rng.integers(0, d_in, 40)]))
    log("wgrad full size: oracle")
    gt_rot = HD.hadamard(np.ascontiguousarray(gb.T), 16, signs)
    xt_rot = HD.hadamard(np.ascontiguousarray(xb.T), 16, signs)
    s_g, s_x = Q.tensor_scale(gt_rot), Q.tensor_scale(xt_rot)
    assert host(qgt[2])[0] == s_g and host(qxt[2])[0] == s_x
    rgt = Q.quantize(gt_rot[ro], s32=s_g, rounding="stochastic", seed=SEED, row_index=ro)
    rxt = Q.quantize(xt_rot[ri], s32=s_x)
    np.testing.assert_array_equal(host(qgt[0])[ro], rgt.codes)
    np.testing.assert_array_equal(host(qxt[1])[ri], rxt.scales)
    a_hat, w_hat = G.operands(rgt, rxt)
    c_ref, bound = G.gemm(a_hat, w_hat)
    ok, worst = G.within_tolerance(dw[np.ix_(ro, ri)], c_ref, bound)
    assert ok.all(), f"{(~ok).sum()} out of tolerance, worst {worst}"
    log(f"wgrad full size worst ratio {worst:.3g}")
