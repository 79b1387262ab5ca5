"""GPU parity of mixfp4_decode_step, the one-launch decode step: A's codes,
scales and tensor scale against the oracle's quantizer bit for bit (compute
mode: s32 from max|A|), C against the oracle's fp64 GEMM of the exactly
dequantized operands within |C - C_ref| <= 1e-5 sum|a w| + 1e-6, and both
against the two-launch path (mixfp4_quantize, then mixfp4_gemm) bit for bit."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gemm as G
from oracle import quant as Q
from tests._gpu import dev_bf16, dev_f32, dev_u8, host, log

pytestmark = pytest.mark.gpu


def _check_c(c, qa, qw, cols=None):
    if cols is not None:
        qw = Q.Quantized(codes=qw.codes[cols], scales=qw.scales[cols], s32=qw.s32, t=None,
                         sf_code=None, si_code=None, delta=None)
        c = c[:, cols]
    a_hat, w_hat = G.operands(qa, qw)
    c_ref, bound = G.gemm(a_hat, w_hat)
    ok, worst = G.within_tolerance(c, c_ref, bound)
    assert ok.all(), f"{(~ok).sum()} elements out of tolerance, worst ratio {worst}"
    return worst


def _step(a_bits, qw_dev):
    import paper_2605_31035_amd as M
    x = dev_bf16(a_bits)
    c, (codes, scales, s32) = M.mixfp4_decode_step(x, qw_dev)
    # the two-launch path on the same input
    rc, rs, rt = M.mixfp4_quantize(x)
    r = M.mixfp4_gemm((rc, rs, rt), qw_dev)
    torch.cuda.synchronize()
    assert torch.equal(codes, rc) and torch.equal(scales, rs) and torch.equal(s32, rt)
    assert torch.equal(c, r)
    return host(c), host(codes), host(scales), host(s32)[0]


@pytest.mark.parametrize("m,n,k", [(16, 300, 4096), (1, 17, 512), (5, 4112, 1024),
                                   (16, 8192, 2048), (11, 12000, 512), (16, 20000, 1024),
                                   (16, 1100, 11008), (2, 700, 256), (16, 900, 4160),
                                   (3, 2000, 192), (9, 5000, 1344)])
def test_shapes(m, n, k):
    """Every column-group width (16 .. 64 columns per workgroup), the K
    splits (four equal shares, two, and four shares that differ by one step:
    k = 11008 is 43 steps of 256, k = 256 one), K tails of 64, 192 and 64
    after 16, 0 and 5 whole steps, ragged m and n, and grids smaller than the
    32 producer workgroups (n = 17: two workgroups)."""
    import paper_2605_31035_amd as M
    a_bits = W.adversarial(m + 3 * n, m, k)
    w_bits = W.adversarial(n + 7, n, k)
    qw = Q.quantize(w_bits)
    qw_dev = (dev_u8(qw.codes), dev_u8(qw.scales), dev_f32(qw.s32))
    log(f"decode step m={m} n={n} k={k}")
    c, codes, scales, s32 = _step(a_bits, qw_dev)
    qa = Q.quantize(a_bits)
    assert np.float32(s32) == np.float32(qa.s32)
    np.testing.assert_array_equal(codes, qa.codes)
    np.testing.assert_array_equal(scales, qa.scales)
    cols = None if n <= 4200 else np.unique(np.concatenate(
        [[0, n - 1], np.random.default_rng(n).integers(0, n, 256)]))
    _check_c(c, qa, qw, cols)
    assert M.decode_step_applies(m, k)


@pytest.mark.parametrize("m,n,k", [(16, 22000, 1024), (3, 28000, 512), (16, 31000, 1024),
                                   (8, 40000, 512), (5, 27940, 512)])
def test_wide_w_column_splits(m, n, k):
    """Wide W: one range of 6 column groups per workgroup, 4 + 3 and 4 + 4
    groups on two sets of waves at once (one workgroup per CU), and 4 groups
    with several workgroups per CU.  W is
    quantized on the device; A's outputs are checked against the oracle bit
    for bit and C on sampled columns."""
    import paper_2605_31035_amd as M
    a_bits = W.adversarial(2 * m + n, m, k)
    w_bits = W.adversarial(5 * n + 3, n, k)
    log(f"decode step wide m={m} n={n} k={k}")
    qw_dev = M.mixfp4_quantize(dev_bf16(w_bits))
    torch.cuda.synchronize()
    c, codes, scales, s32 = _step(a_bits, qw_dev)
    qa = Q.quantize(a_bits)
    assert np.float32(s32) == np.float32(qa.s32)
    np.testing.assert_array_equal(codes, qa.codes)
    np.testing.assert_array_equal(scales, qa.scales)
    cols = np.unique(np.concatenate([[0, n - 1], np.arange(0, n, 1792)[:40],
                                     np.random.default_rng(n).integers(0, n, 96)]))
    qw = Q.quantize(w_bits[cols], s32=Q.tensor_scale(w_bits))
    np.testing.assert_array_equal(host(qw_dev[0])[cols], qw.codes)
    _check_c(c[:, cols], qa, qw)


def test_decode_workload_full_size():
    """The decode workload in the launch configuration the benchmark times:
    A[16,8192] quantized in the step, W[28672,8192] quantized before."""
    wl = W.decode()
    a_bits, w_bits = wl.tensors["A"], wl.tensors["W"]
    import paper_2605_31035_amd as M
    log("decode workload: quantize W on the device")
    qw_dev = M.mixfp4_quantize(dev_bf16(w_bits))
    torch.cuda.synchronize()
    c, codes, scales, s32 = _step(a_bits, qw_dev)
    qa = Q.quantize(a_bits)
    assert np.float32(s32) == np.float32(qa.s32)
    np.testing.assert_array_equal(codes, qa.codes)
    np.testing.assert_array_equal(scales, qa.scales)
    cols = np.unique(np.concatenate([[0, w_bits.shape[0] - 1],
                                     np.random.default_rng(3).integers(0, w_bits.shape[0], 96)]))
    qw = Q.quantize(w_bits[cols], s32=Q.tensor_scale(w_bits))
    np.testing.assert_array_equal(host(qw_dev[0])[cols], qw.codes)
    worst = _check_c(c[:, cols], qa, qw)
    log(f"decode workload ok, worst ratio {worst:.3g}")


def test_calls_in_a_row_and_sync_reset():
    """Three steps in a row on one sync buffer with different activations
    (the launch returns the counters to zero), one of them all zeros
    (s32 = 1, every block the E1M2 zero, C = 0)."""
    import paper_2605_31035_amd as M
    m, n, k = 16, 3000, 2048
    w_bits = W.adversarial(5, n, k)
    qw = Q.quantize(w_bits)
    qw_dev = (dev_u8(qw.codes), dev_u8(qw.scales), dev_f32(qw.s32))
    sync = torch.zeros(4, dtype=torch.int32, device="cuda")
    for seed in (1, 2, 0):
        a_bits = W.adversarial(seed, m, k) if seed else np.zeros((m, k), dtype=np.uint16)
        c, (codes, scales, s32) = M.mixfp4_decode_step(dev_bf16(a_bits), qw_dev, sync=sync)
        torch.cuda.synchronize()
        assert int(sync.abs().sum().item()) == 0
        qa = Q.quantize(a_bits)
        np.testing.assert_array_equal(host(codes), qa.codes)
        np.testing.assert_array_equal(host(scales), qa.scales)
        assert np.float32(host(s32)[0]) == np.float32(qa.s32)
        if seed == 0:
            assert np.float32(qa.s32) == np.float32(1.0)
            assert np.all(host(scales) == 0x80) and np.all(host(c) == 0)
        else:
            _check_c(host(c), qa, qw)


def test_rejects():
    import paper_2605_31035_amd as M
    w = M.mixfp4_quantize(torch.zeros((8, 512), dtype=torch.bfloat16, device="cuda"))
    for shape in ((17, 512), (4, 96), (0, 512)):
        with pytest.raises(ValueError):
            M.mixfp4_decode_step(torch.zeros(shape, dtype=torch.bfloat16, device="cuda"), w)
    with pytest.raises(ValueError):
        M.mixfp4_decode_step(torch.zeros((4, 1024), dtype=torch.bfloat16, device="cuda"), w)
