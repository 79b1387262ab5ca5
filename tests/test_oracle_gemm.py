"""Pins for oracle.gemm: the fp64 matmul of exactly dequantized operands
against a rational dot product (App. B.1), integer-valued operands where the
result is exact, and the tolerance helper."""
from fractions import Fraction

import numpy as np

from oracle import exact as E
from oracle import gemm as G
from oracle import quant as Q
from workloads import f32_to_bf16_bits


def test_matches_rational_dot():
    rng = np.random.default_rng(11)
    a = f32_to_bf16_bits(rng.standard_t(3, (4, 48)).astype(np.float32))
    w = f32_to_bf16_bits((rng.standard_normal((5, 48)) * 0.02).astype(np.float32))
    qa, qw = Q.quantize(a), Q.quantize(w)
    a_hat, w_hat = G.operands(qa, qw)
    c, bound = G.gemm(a_hat, w_hat)
    sa, sw = Fraction(float(qa.s32)), Fraction(float(qw.s32))
    for m in range(4):
        for n in range(5):
            terms = []
            for kk in range(48):
                na = (int(qa.codes[m, kk // 2]) >> (4 * (kk % 2))) & 15
                nw = (int(qw.codes[n, kk // 2]) >> (4 * (kk % 2))) & 15
                va = sa * E.decode_value(na, int(qa.scales[m, kk // 16]))
                vw = sw * E.decode_value(nw, int(qw.scales[n, kk // 16]))
                terms.append(va * vw)
            exact = sum(terms, Fraction(0))
            assert abs(Fraction(c[m, n]) - exact) <= Fraction(1, 10 ** 12) * sum(abs(t) for t in terms)
            assert bound[m, n] == float(sum(abs(t) for t in terms)) or abs(bound[m, n] - float(sum(abs(t) for t in terms))) <= 1e-12 * bound[m, n]


def test_integer_operands_exact():
    rng = np.random.default_rng(12)
    # on-grid INT4 blocks with s8 = 1 and s32 = 1: values are small integers
    a = rng.integers(-7, 8, (8, 64)).astype(np.float32)
    w = rng.integers(-7, 8, (6, 64)).astype(np.float32)
    a.reshape(-1, 16)[:, 0] = 7
    w.reshape(-1, 16)[:, 0] = 7
    qa = Q.quantize(f32_to_bf16_bits(a), s32=1.0)
    qw = Q.quantize(f32_to_bf16_bits(w), s32=1.0)
    a_hat, w_hat = G.operands(qa, qw)
    assert np.array_equal(a_hat, a) and np.array_equal(w_hat, w)
    c, _ = G.gemm(a_hat, w_hat)
    assert np.array_equal(c, a.astype(np.int64) @ w.astype(np.int64).T)


def test_tolerance_helper():
    c_ref = np.array([[1.0, -2.0]])
    bound = np.array([[10.0, 10.0]])
    ok, worst = G.within_tolerance(c_ref + np.array([[1e-4 + 1e-6 - 1e-9, 0.0]]), c_ref, bound)
    assert ok.all() and worst < 1
    ok, worst = G.within_tolerance(c_ref + np.array([[2e-4, 0.0]]), c_ref, bound)
    assert not ok.all() and worst > 1
