"""mixfp4_gemm_noalloc (the GEMM whose workspace is the library's static
device array) through the C ABI: equal to mixfp4_gemm_ws with a caller
workspace, bit for bit, and within the oracle's tolerance, on two calls in a
row, the second with a smaller problem (the array keeps the first call's
contents); shapes beyond the array are rejected before anything is enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import workloads as W
from oracle import gemm as G
from oracle import quant as Q
from tests._gpu import dev_f32, dev_u8, host, log

pytestmark = pytest.mark.gpu


def _dev(q):
    return (dev_u8(q.codes), dev_u8(q.scales), dev_f32(q.s32))


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _noalloc(a, w, m, n, k):
    from paper_2605_31035_amd import _lib
    c = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
    st = _lib.lib.mixfp4_gemm_noalloc(_p(a[0]), _p(a[1]), _p(a[2]), _p(w[0]), _p(w[1]), _p(w[2]),
                                      m, n, k, _p(c),
                                      ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    return st, c


def _check(c, qa, qw):
    a_hat, w_hat = G.operands(qa, qw)
    c_ref, bound = G.gemm(a_hat, w_hat)
    ok, worst = G.within_tolerance(c, c_ref, bound)
    assert ok.all(), f"{(~ok).sum()} elements out of tolerance, worst ratio {worst}"


def test_noalloc_matches_workspace_path_twice():
    import paper_2605_31035_amd as M
    from paper_2605_31035_amd import _lib
    cap = _lib.lib.mixfp4_gemm_noalloc_max_bytes()
    assert cap == 64 << 20
    for (m, n, k) in [(1024, 2048, 4096), (300, 520, 1056)]:     # second call smaller
        assert 0 < M.mixfp4_gemm_workspace_size(m, n, k) <= cap
        qa = Q.quantize(W.adversarial(m + 3 * k, m, k))
        qw = Q.quantize(W.adversarial(n + 7 * k, n, k))
        a, w = _dev(qa), _dev(qw)
        log(f"noalloc m={m} n={n} k={k}")
        st, c = _noalloc(a, w, m, n, k)
        assert st == 0
        ref = M.mixfp4_gemm(a, w, workspace=True)
        torch.cuda.synchronize()
        assert torch.equal(c, ref)
        if m * n <= 300 * 520:
            _check(host(c), qa, qw)
        else:
            rows, cols = np.arange(0, m, 37), np.arange(0, n, 41)
            sub = lambda q, r: Q.Quantized(codes=q.codes[r], scales=q.scales[r], s32=q.s32,  # noqa
                                           t=None, sf_code=None, delta=None, si_code=None)
            _check(host(c)[np.ix_(rows, cols)], sub(qa, rows), sub(qw, cols))


def test_noalloc_rejects_beyond_the_array_and_keeps_decode_shapes():
    import paper_2605_31035_amd as M
    m, n, k = 4096, 4096, 8192        # workspace 128 MiB > 64 MiB
    assert M.mixfp4_gemm_workspace_size(m, n, k) > (64 << 20)
    codes = torch.zeros((max(m, n), k // 2), dtype=torch.uint8, device="cuda")
    scales = torch.zeros((max(m, n), k // 16), dtype=torch.uint8, device="cuda")
    st, c = _noalloc((codes, scales, None), (codes, scales, None), m, n, k)
    assert st == 6                    # MIXFP4_ERR_SCRATCH
    torch.cuda.synchronize()
    assert torch.isnan(c).all()       # nothing was enqueued
    # a decode shape needs no workspace: the fused kernel, as mixfp4_gemm
    qa = Q.quantize(W.adversarial(5, 16, 2048))
    qw = Q.quantize(W.adversarial(6, 300, 2048))
    a, w = _dev(qa), _dev(qw)
    st, c = _noalloc(a, w, 16, 300, 2048)
    assert st == 0
    ref = M.mixfp4_gemm(a, w)
    torch.cuda.synchronize()
    assert torch.equal(c, ref)
