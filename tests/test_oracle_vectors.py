"""Pins for oracle.quant / oracle.gemm against the hand-worked fixtures in
tests/golden (derived on paper from Algorithm 1, Table 1, App. B.1-B.3)."""
from fractions import Fraction

import numpy as np

from oracle import exact as E
from oracle import gemm as G
from oracle import quant as Q
from tests._golden import handworked_blocks, handworked_gemm
from workloads import f32_to_bf16_bits


def _blocks():
    cases = handworked_blocks()
    x = np.stack([c["block"] for c in cases])
    return cases, f32_to_bf16_bits(x)


def test_handworked_blocks_fast_oracle():
    cases, bits = _blocks()
    q = Q.quantize(bits, s32=1.0)
    for i, c in enumerate(cases):
        assert q.scales[i, 0] == c["scale"], i
        assert bytes(q.codes[i]) == c["codes"], i
        assert int(q.t[i, 0]) == c["t"]
        sf = Fraction(float(Q.F.e4m3_decode(q.sf_code[i, 0])))
        si = Fraction(float(Q.F.e4m3_decode(q.si_code[i, 0])))
        assert (sf, si) == c["sigma"], i
        assert Fraction(float(q.delta[i, 0])) == c["err"][0] - c["err"][1], i


def test_handworked_blocks_exact_oracle():
    cases, bits = _blocks()
    for i, c in enumerate(cases):
        sb, nibs, ef, ei = E.quantize_block(bits[i], Fraction(1))
        assert sb == c["scale"]
        assert bytes(nibs[j] | (nibs[j + 1] << 4) for j in range(0, 16, 2)) == c["codes"]
        assert (ef, ei) == c["err"]


def test_handworked_dot():
    g = handworked_gemm()
    bits = f32_to_bf16_bits(np.array([g["a"], g["w"]], dtype=np.float32))
    qa = Q.quantize(bits[:1], s32=1.0)
    qw = Q.quantize(bits[1:], s32=1.0)
    a_hat, w_hat = G.operands(qa, qw)
    assert a_hat[0].tolist() == g["a_decoded"]
    assert w_hat[0].tolist() == g["w_decoded"]
    c, bound = G.gemm(a_hat, w_hat)
    assert c[0, 0] == g["c"][0]
    assert bound[0, 0] == sum(abs(x * y) for x, y in zip(g["a_decoded"], g["w_decoded"]))


def test_dequantize_handworked():
    cases, bits = _blocks()
    q = Q.quantize(bits, s32=1.0)
    d = Q.dequantize(q.codes, q.scales)
    # the [6,4,3,...] block decodes to its grid values (ties resolved to even codes)
    assert d[4, :10].tolist() == [6, 4, 3, 2, 1.5, 1, 0.5, 0, 1, -1]
    assert d[0, 0] == 6 and d[1, 0] == 7
    assert np.all(d[5] == 0)
