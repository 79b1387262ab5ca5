"""GPU parity of mixfp4_quantize_variant / mixfp4_dequantize_variant (other
candidate sets and block sizes: Sec. 2.3-2.4, Fig. 3, Table 5) against
``oracle.variants``: codes, scale bytes, chosen indices and s32 bit-exact,
dequantized values bit-exact."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import quant as Q
from oracle import variants as V
from tests._gpu import dev_bf16, dev_f32, host, log

pytestmark = pytest.mark.gpu

MASKS = {1: ("e2m1",), 2: ("e1m2",), 3: ("e2m1", "e1m2"), 4: ("e3m0",), 5: ("e2m1", "e3m0"),
         6: ("e1m2", "e3m0"), 7: ("e2m1", "e1m2", "e3m0")}


def _mixed(seed, rows, k):
    rng = np.random.default_rng(seed)
    x = rng.standard_t(3, (rows, k)).astype(np.float32)
    x[0, : min(k, 64)] = -0.0
    x[1, : min(k, 32)] = np.arange(min(k, 32)) * 0.25
    x[2] = 2.0 ** rng.integers(-9, 6, k) * rng.choice([-1, 1], k)
    x[3] = rng.integers(-7, 8, k)
    x[4, ::3] = 48.0
    x[5] *= 1e-30
    return W.f32_to_bf16_bits(x)


def _check(bits, block, mask, s32=None, ldx_pad=0, label=""):
    import paper_2605_31035_amd as M
    cands = MASKS[mask]
    log(f"variant {label} shape={bits.shape} block={block} set={cands} s32={s32} pad={ldx_pad}")
    x = dev_bf16(bits)
    if ldx_pad:
        big = torch.zeros((bits.shape[0], bits.shape[1] + ldx_pad), dtype=torch.bfloat16,
                          device="cuda")
        big[:, : bits.shape[1]] = x
        x = big[:, : bits.shape[1]]
    q = M.mixfp4_quantize_variant(x, block, cands, None if s32 is None else dev_f32(s32))
    ref = V.quantize_variant(bits, block, cands, s32)
    assert host(q.s32)[0] == ref.s32
    np.testing.assert_array_equal(host(q.scales), ref.scales)
    np.testing.assert_array_equal(host(q.fmt), ref.fmt)
    np.testing.assert_array_equal(host(q.codes), ref.codes)
    d = host(M.mixfp4_dequantize_variant(q))
    np.testing.assert_array_equal(d, V.dequantize(ref))
    if len(cands) < 3:
        np.testing.assert_array_equal(host(M.mixfp4_dequantize_variant(q, use_fmt=False)), d)
    return q, ref


@pytest.mark.parametrize("block", [8, 16, 32, 64])
@pytest.mark.parametrize("mask", sorted(MASKS))
def test_every_set_and_block_size(block, mask):
    _check(_mixed(block + mask, 24, 256), block, mask, label="mixed")
    _check(W.adversarial(block * mask, 7, 192), block, mask, label="adversarial")


@pytest.mark.parametrize("block", [8, 32, 64])
@pytest.mark.parametrize("mask", [3, 5, 7])
def test_given_scales_strides_and_clamping(block, mask):
    """Given tensor scales, including ones far below max|X| / 2688 (block
    scales clamped at 448, the compensated comparison) and above it, strided
    rows and ragged row counts."""
    bits = _mixed(7 * block + mask, 13, 128)
    amax = float(np.abs(Q.bf16_to_f32(bits)).max())
    for s32 in (np.float32(0.37), np.float32(amax / 2688 / 1000), np.float32(amax / 20),
                np.float32(2.0 ** -100)):
        _check(bits, block, mask, s32=s32, label="given")
    _check(bits, block, mask, ldx_pad=8, label="ldx=k+8")
    _check(bits, block, mask, s32=np.float32(1.5), ldx_pad=64, label="ldx=k+64 given")


def test_mixfp4_pair_equals_mixfp4_quantize():
    """{E2M1, E1M2} at block 16 is MixFP4: the variant kernel and the
    product quantizer agree bit for bit on a prefill-shaped activation."""
    import paper_2605_31035_amd as M
    bits = W.prefill_7b().tensors["A"][:512]
    x = dev_bf16(bits)
    q = M.mixfp4_quantize_variant(x, 16, ("e2m1", "e1m2"))
    c, s, t = M.mixfp4_quantize(x)
    torch.cuda.synchronize()
    assert torch.equal(q.codes, c) and torch.equal(q.scales, s) and torch.equal(q.s32, t)


def test_empty_and_zero():
    import paper_2605_31035_amd as M
    for block, mask in ((8, 7), (64, 5)):
        q = M.mixfp4_quantize_variant(torch.zeros((0, 128), dtype=torch.bfloat16, device="cuda"),
                                      block, MASKS[mask])
        assert host(q.s32)[0] == 1.0
        _check(np.zeros((3, 128), np.uint16), block, mask, label="zeros")


@pytest.mark.parametrize("block,mask", [(32, 5), (64, 7), (8, 3)])
def test_full_size_sampled_rows(block, mask):
    """The large activation A[16384, 8192] in the launch configuration the
    benchmark times; s32 exact and sampled rows against the oracle."""
    import paper_2605_31035_amd as M
    bits = W.large(tensors=("A",)).tensors["A"]
    q = M.mixfp4_quantize_variant(dev_bf16(bits), block, MASKS[mask])
    rows = np.unique(np.concatenate([[0, bits.shape[0] - 1],
                                     np.random.default_rng(block).integers(0, bits.shape[0], 24)]))
    s32 = Q.tensor_scale(bits)
    assert host(q.s32)[0] == s32
    ref = V.quantize_variant(bits[rows], block, MASKS[mask], s32)
    np.testing.assert_array_equal(host(q.codes)[rows], ref.codes)
    np.testing.assert_array_equal(host(q.scales)[rows], ref.scales)
    np.testing.assert_array_equal(host(q.fmt)[rows], ref.fmt)
    log(f"full size block={block} set={MASKS[mask]} ok")
