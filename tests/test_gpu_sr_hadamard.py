"""GPU parity of stochastic rounding (App. D), the block-diagonal Hadamard
transform, and rotate-then-quantize, against the CPU oracle: bf16 outputs,
codes, scale bytes and s32 bit-exact."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import hadamard as HD
from oracle import quant as Q
from tests._gpu import dev_bf16, dev_f32, host, log

pytestmark = pytest.mark.gpu

SEED = 0xDEADBEEF12345678
OFFSET = (1 << 40) + 7


def _padded(bits, pad):
    x = dev_bf16(bits)
    if pad:
        rows, k = bits.shape
        big = torch.zeros((rows, k + pad), dtype=torch.bfloat16, device="cuda")
        big[:, :k] = x
        x = big[:, :k]
    return x


def _signs_dev(signs):
    return None if signs is None else torch.tensor(np.where(signs < 0, -1, 1).astype(np.int8),
                                                   device="cuda")


def _check_quant(got, ref, label):
    codes, scales, s = got
    torch.cuda.synchronize()
    assert host(s)[0] == ref.s32, (label, host(s)[0], ref.s32)
    np.testing.assert_array_equal(host(scales), ref.scales, err_msg=label)
    np.testing.assert_array_equal(host(codes), ref.codes, err_msg=label)


# ---------------------------------------------------------------- stochastic rounding

@pytest.mark.parametrize("mode,omode", [("mixfp4", "select"), ("e2m1", "e2m1"), ("e1m2", "e1m2"),
                                        ("four_six", "four_six")])
@pytest.mark.parametrize("rows,k,s32,pad", [(3, 48, None, 0), (64, 4096, None, 0),
                                            (65, 4096, None, 0), (257, 80, 0.37, 0),
                                            (33, 64, None, 8), (300, 1024, 1.5, 24)])
def test_stochastic_rounding(mode, omode, rows, k, s32, pad):
    """Small one-launch path (COMPUTE, <= 2^18 elements), two-pass path,
    given s32, strided rows; seed and offset with high words set."""
    import paper_2605_31035_amd as M
    bits = W.adversarial(rows + k, rows, k)
    label = f"sr {mode} {rows}x{k} s32={s32} pad={pad}"
    log(label)
    ts = None if s32 is None else dev_f32(s32)
    got = M.mixfp4_quantize(_padded(bits, pad), ts, mode=mode, rounding="stochastic", seed=SEED,
                            offset=OFFSET)
    ref = Q.quantize(bits, s32=s32, mode=omode, rounding="stochastic", seed=SEED, offset=OFFSET)
    _check_quant(got, ref, label)


def test_stochastic_rounding_streams_differ_and_repeat():
    import paper_2605_31035_amd as M
    bits = W.adversarial(5, 128, 512)
    x = dev_bf16(bits)
    a = host(M.mixfp4_quantize(x, rounding="stochastic", seed=1, offset=0)[0])
    b = host(M.mixfp4_quantize(x, rounding="stochastic", seed=1, offset=0)[0])
    c = host(M.mixfp4_quantize(x, rounding="stochastic", seed=1, offset=1)[0])
    d = host(M.mixfp4_quantize(x, rounding="stochastic", seed=2, offset=0)[0])
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c) and not np.array_equal(a, d)


def test_stochastic_rounding_full_size():
    """The 7B-class prefill activation (2048 x 4096), sampled rows against the
    oracle under the GPU-independent s32 of the whole tensor."""
    import paper_2605_31035_amd as M
    wl = W.get("prefill_7b", tensors=("A",))
    bits = wl.tensors["A"]
    log("sr full size prefill A")
    codes, scales, s = M.mixfp4_quantize(dev_bf16(bits), rounding="stochastic", seed=SEED,
                                         offset=3)
    torch.cuda.synchronize()
    s32 = Q.tensor_scale(bits)
    assert host(s)[0] == s32
    rows = np.unique(np.concatenate([[0, bits.shape[0] - 1],
                                     np.random.default_rng(4).integers(0, bits.shape[0], 96)]))
    # the draws of a block depend on its global index: quantize the full rows'
    # blocks at their own indices by running the oracle on whole rows in place
    ref = Q.quantize(bits[rows], s32=s32, rounding="stochastic", seed=SEED, offset=3,
                     row_index=rows)
    np.testing.assert_array_equal(host(scales)[rows], ref.scales)
    np.testing.assert_array_equal(host(codes)[rows], ref.codes)


# ---------------------------------------------------------------- Hadamard transform

def _hadamard_cases(b, rng):
    rows = 37
    x = rng.standard_t(3, (rows, 4 * b)).astype(np.float32)
    x[0] = 0.0
    x[1, :b] = -0.0
    x[2, : b // 2] *= np.float32(2.0 ** 20)          # wide (in-contract) spread
    x[3, 5] = np.float32(3e38)                       # overflow in its block
    x[4, :] *= np.float32(2.0 ** -125)               # subnormal outputs
    x[5, ::7] = 0.0
    return W.f32_to_bf16_bits(x)


@pytest.mark.parametrize("b", HD.BLOCKS)
@pytest.mark.parametrize("with_signs", [False, True])
def test_hadamard_transform(b, with_signs):
    import paper_2605_31035_amd as M
    rng = np.random.default_rng(b + 7 * with_signs)
    bits = _hadamard_cases(b, rng)
    signs = rng.choice([-1, 1], size=b) if with_signs else None
    log(f"hadamard b={b} signs={with_signs} shape={bits.shape}")
    ref = HD.hadamard(bits, b, signs)
    for pad in (0, 8):
        y = M.mixfp4_hadamard(_padded(bits, pad), b, _signs_dev(signs))
        torch.cuda.synchronize()
        got = host(y.view(torch.int16)).view(np.uint16)
        np.testing.assert_array_equal(got, ref, err_msg=f"b={b} pad={pad}")


@pytest.mark.parametrize("b", [32, 128])
def test_hadamard_near_midpoints(b):
    """Outputs built to lie within about 2^-60 of a bf16 rounding midpoint
    (the exact square comparison decides them)."""
    import paper_2605_31035_amd as M
    from tests.test_oracle_hadamard import _split_bf16
    import decimal
    decimal.getcontext().prec = 120
    rows = []
    for mant in range(129, 256, 3):
        for side in (0, 1):
            mid = (2 * mant + 1) / 2 * 2.0 ** -7
            target = decimal.Decimal(mid) * decimal.Decimal(2) ** 20 * decimal.Decimal(b).sqrt()
            S = int(target.to_integral_value(rounding=decimal.ROUND_FLOOR)) + side
            x = np.zeros(b, np.float64)
            parts = _split_bf16(S, 8)
            x[: len(parts)] = parts
            rows.append(x)
    bits = W.f32_to_bf16_bits(np.array(rows).astype(np.float32))
    ref = HD.hadamard(bits, b)
    log(f"hadamard near midpoints b={b} rows={len(rows)}")
    got = host(M.mixfp4_hadamard(dev_bf16(bits), b).view(torch.int16)).view(np.uint16)
    np.testing.assert_array_equal(got, ref)


def test_hadamard_full_size():
    """Config-3-sized activation (4096 x 4096) with 128-blocks and random
    signs, checked in full."""
    import paper_2605_31035_amd as M
    rng = np.random.default_rng(11)
    x = rng.standard_t(3, (4096, 4096)).astype(np.float32)
    bits = W.f32_to_bf16_bits(x)
    signs = rng.choice([-1, 1], size=128)
    log("hadamard full size 4096x4096 b=128")
    got = host(M.mixfp4_hadamard(dev_bf16(bits), 128, _signs_dev(signs)).view(torch.int16))
    ref = HD.hadamard(bits, 128, signs)
    np.testing.assert_array_equal(got.view(np.uint16), ref)


# ---------------------------------------------------------------- rotate, then quantize

@pytest.mark.parametrize("b", [16, 64, 128, 256])
@pytest.mark.parametrize("mode,omode", [("mixfp4", "select"), ("e2m1", "e2m1")])
@pytest.mark.parametrize("rounding", ["nearest", "stochastic"])
@pytest.mark.parametrize("s32", [None, 0.25])
def test_rotate_then_quantize(b, mode, omode, rounding, s32):
    import paper_2605_31035_amd as M
    rng = np.random.default_rng(b)
    rows, k = 70, 2 * 256
    bits = W.adversarial(b + 100, rows, k)
    signs = rng.choice([-1, 1], size=b)
    label = f"rht b={b} {mode} {rounding} s32={s32}"
    log(label)
    ts = None if s32 is None else dev_f32(s32)
    got = M.mixfp4_quantize(_padded(bits, 8 if s32 else 0), ts, mode=mode, rounding=rounding,
                            seed=SEED, offset=OFFSET, hadamard_block=b,
                            hadamard_signs=_signs_dev(signs))
    rot = HD.hadamard(bits, b, signs)
    ref = Q.quantize(rot, s32=s32, mode=omode, rounding=rounding, seed=SEED, offset=OFFSET)
    _check_quant(got, ref, label)


def test_rotate_then_quantize_full_size():
    """The 7B-class prefill activation rotated with 128-blocks then quantized
    (COMPUTE mode: s32 from the rotated tensor), checked in full."""
    import paper_2605_31035_amd as M
    wl = W.get("prefill_7b", tensors=("A",))
    bits = wl.tensors["A"]
    rng = np.random.default_rng(12)
    signs = rng.choice([-1, 1], size=128)
    log("rht full size prefill A b=128")
    got = M.mixfp4_quantize(dev_bf16(bits), hadamard_block=128, hadamard_signs=_signs_dev(signs))
    ref = Q.quantize(HD.hadamard(bits, 128, signs))
    _check_quant(got, ref, "rht full size")
