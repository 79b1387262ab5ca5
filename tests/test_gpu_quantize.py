"""GPU parity of mixfp4_quantize / mixfp4_dequantize against the CPU oracle:
codes, scale bytes and s32 bit-exact, dequantized values bit-exact."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import quant as Q
from tests._golden import handworked_blocks
from tests._gpu import dev_bf16, dev_f32, dev_u8, gpu_quantize, host, log

pytestmark = pytest.mark.gpu


def _assert_same(bits, s32=None, ldx_pad=0, label=""):
    log(f"quantize {label} shape={bits.shape} s32={s32} pad={ldx_pad}")
    codes, scales, s = gpu_quantize(bits, s32, ldx_pad)
    ref = Q.quantize(bits, s32=s32)
    assert host(s)[0] == ref.s32, (host(s)[0], ref.s32)
    np.testing.assert_array_equal(host(scales), ref.scales)
    np.testing.assert_array_equal(host(codes), ref.codes)
    return codes, scales, s, ref


def test_handworked_blocks():
    cases = handworked_blocks()
    bits = W.f32_to_bf16_bits(np.stack([c["block"] for c in cases]))
    codes, scales, _, _ = _assert_same(bits, s32=1.0, label="handworked")
    for i, c in enumerate(cases):
        assert host(scales)[i, 0] == c["scale"]
        assert bytes(host(codes)[i]) == c["codes"]


def test_tiny_workload_and_dequant():
    import paper_2605_31035_amd as M
    wl = W.tiny()
    for name, bits in wl.tensors.items():
        codes, scales, s, ref = _assert_same(bits, label=f"tiny.{name}")
        d = host(M.mixfp4_dequantize(codes, scales, s))
        np.testing.assert_array_equal(d, Q.dequantize(ref.codes, ref.scales, ref.s32))
        d1 = host(M.mixfp4_dequantize(codes, scales, None))
        np.testing.assert_array_equal(d1, Q.dequantize(ref.codes, ref.scales, None))


@pytest.mark.parametrize("rows,k,seed", [(1, 16, 0), (3, 48, 1), (257, 80, 2), (64, 4096, 3), (1000, 272, 4)])
def test_adversarial(rows, k, seed):
    bits = W.adversarial(seed, rows, k)
    _assert_same(bits, label="adversarial")
    _assert_same(bits, s32=np.float32(0.37), label="adversarial/given")


def test_strided_rows():
    bits = W.adversarial(9, 33, 64)
    _assert_same(bits, ldx_pad=8, label="ldx=k+8")
    _assert_same(bits, ldx_pad=64, s32=1.5, label="ldx=k+64 given")


def test_near_midpoints():
    from oracle import formats as F
    rows = []
    for s8 in F.E4M3_VALUES[1:126:3]:
        for grid, top in ((F.F_GRID, 6.0), (F.I_GRID, 7.0)):
            mids = (grid[:-1] + grid[1:]) / 2
            blk = np.zeros(16, np.float32)
            vals = ([top * s8] + list(mids * s8) + list(grid[1:] * s8))[:16]
            blk[:len(vals)] = np.array(vals, np.float32)
            rows.append(blk)
            rows.append(-blk)
    bits = W.f32_to_bf16_bits(np.stack(rows))
    for b in (bits, np.where(bits & 0x7FFF, bits + 1, bits).astype(np.uint16)):
        for s in (1.0, 1 + 2 ** -23, 1 - 2 ** -24, 1 + 5 * 2 ** -23, 0.75 - 2 ** -25):
            _assert_same(b, s32=np.float32(s), label="near-midpoint")


@pytest.mark.parametrize("exp,s32", [
    (-100, None), (-60, None), (100, None), (112, None),
    (-100, 1.3 * 2.0 ** -100), (112, 1.1 * 2.0 ** 121), (-125, 1.5 * 2.0 ** -140)])
def test_extreme_tensor_scales(exp, s32):
    """Data scaled by 2^exp and tensor scales far from 1 (down to an fp32
    subnormal s32): below 2^-90 and above 2^120 the kernel rescales X and s32
    by 2^64 or 2^-64 before dividing; in between it divides directly."""
    f = W.bf16_bits_to_f32(W.adversarial(200 + exp, 48, 256)).astype(np.float64) * 2.0 ** exp
    bits = W.f32_to_bf16_bits(f.astype(np.float32))
    given = None if s32 is None else np.float32(s32)
    _assert_same(bits, s32=given, label=f"2^{exp} data")


@pytest.mark.parametrize("exp", [-20, 0, 7])
def test_tensor_scale_fallback(exp):
    """The tensor scales on which the two-term division misses the exact
    quotient for one bf16 mantissa (census in test_division_step): the
    launch-time check must route them to Markstein's step.  Each tensor holds
    that mantissa at several exponents and both signs, among adversarial
    blocks."""
    from tests.test_division_step import FALLBACK_PAIRS
    for s_bits, x_bits in FALLBACK_PAIRS:
        s32 = np.float32(np.uint32(s_bits).view(np.float32) * np.float32(2.0 ** exp))
        a = np.uint32(x_bits).view(np.float32) * np.float32(2.0 ** exp)
        bits = W.adversarial(s_bits & 0xFFFF, 24, 64)
        special = np.array([a * np.float32(2.0 ** j) * sg for j in range(-4, 4) for sg in (1, -1)],
                           np.float32)
        bits[:, 0] = W.f32_to_bf16_bits(special[np.arange(24) % 16])
        bits[::3, 16:32] = W.f32_to_bf16_bits(special)
        _assert_same(bits, s32=s32, label=f"fallback s32=0x{s_bits:08x}*2^{exp}")


@pytest.mark.parametrize("rows,k,pad", [(64, 4096, 0), (65, 4096, 0), (1, 1 << 18, 0),
                                        (16, 8192, 0), (3, 48, 8), (100, 1024, 64),
                                        (2049, 8192, 0)])
def test_small_and_large_compute_paths(rows, k, pad):
    """Tensors of at most 2^18 elements get their tensor scale and codes in one
    launch (every workgroup reduces max|X| itself); larger ones take the
    amax / reduce / quantize sequence.  Both sides of the threshold, strided
    rows included, must give the oracle's bits."""
    bits = W.adversarial(rows * 7 + k, rows, k)
    _assert_same(bits, ldx_pad=pad, label=f"compute path {rows}x{k}")


@pytest.mark.parametrize("mode,omode", [("mixfp4", "select"), ("e2m1", "e2m1"),
                                        ("e1m2", "e1m2"), ("four_six", "four_six")])
@pytest.mark.parametrize("rounding", ["nearest", "stochastic"])
@pytest.mark.parametrize("rows,k,pad", [(65, 4096, 0), (601, 1008, 24), (4096, 4096, 0)])
def test_compute_mode_matrix(mode, omode, rounding, rows, k, pad):
    """The amax / reduce / quantize sequence (tensor scale computed, above the
    one-launch size): every format mode and both roundings, ragged block
    counts and strided rows; 4096 x 4096 has more blocks than resident
    threads, so each thread takes several (checked on sampled rows there, in
    full elsewhere)."""
    import paper_2605_31035_amd as M
    bits = W.adversarial(rows + 5 * k, rows, k)
    label = f"compute {mode} {rounding} {rows}x{k} pad={pad}"
    log(label)
    x = dev_bf16(bits)
    if pad:
        big = torch.zeros((rows, k + pad), dtype=torch.bfloat16, device="cuda")
        big[:, :k] = x
        x = big[:, :k]
    seed = 0x5EED0F05ED
    codes, scales, s = M.mixfp4_quantize(x, mode=mode, rounding=rounding, seed=seed, offset=3)
    torch.cuda.synchronize()
    s_ref = Q.tensor_scale(bits)
    assert host(s)[0] == s_ref, label
    sel = np.arange(rows) if rows * k <= (1 << 20) else _sampled_rows(np.random.default_rng(1), rows)
    # the selected rows with the full tensor's s32, numbered as in the full
    # tensor (stochastic rounding draws by block index)
    ref = Q.quantize(bits[sel], s32=s_ref, mode=omode, rounding=rounding, seed=seed, offset=3,
                     row_index=sel)
    idx = torch.from_numpy(sel).to("cuda")
    np.testing.assert_array_equal(host(scales.index_select(0, idx)), ref.scales, err_msg=label)
    np.testing.assert_array_equal(host(codes.index_select(0, idx)), ref.codes, err_msg=label)


@pytest.mark.parametrize("mode", ["e2m1", "e1m2", "four_six"])
@pytest.mark.parametrize("rows,k,s32", [(3, 48, None), (64, 4096, None), (65, 4096, None),
                                        (257, 80, 0.37), (1000, 272, None)])
def test_forced_format_modes(mode, rows, k, s32):
    """E2M1-only (NVFP4), E1M2-only (INT4) and 4/6 modes, small one-launch and
    large paths, computed and given tensor scales: the oracle's bits."""
    import paper_2605_31035_amd as M
    bits = W.adversarial(rows + 3 * k, rows, k)
    given = None if s32 is None else np.float32(s32)
    log(f"quantize forced {mode} {rows}x{k} s32={given}")
    x = dev_bf16(bits)
    ts = None if given is None else dev_f32(given)
    codes, scales, s = M.mixfp4_quantize(x, ts, mode=mode)
    torch.cuda.synchronize()
    ref = Q.quantize(bits, s32=given, mode=mode)
    assert host(s)[0] == ref.s32
    np.testing.assert_array_equal(host(scales), ref.scales)
    np.testing.assert_array_equal(host(codes), ref.codes)


def test_empty_inputs():
    import paper_2605_31035_amd as M
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    codes, scales, s = M.mixfp4_quantize(x)
    torch.cuda.synchronize()
    assert codes.shape == (0, 32) and host(s)[0] == 1.0
    x = torch.zeros((5, 64), dtype=torch.bfloat16, device="cuda")
    codes, scales, s = M.mixfp4_quantize(x)
    assert host(s)[0] == 1.0 and np.all(host(scales) == 0x80) and np.all(host(codes) == 0)


def test_deterministic():
    bits = W.adversarial(21, 512, 1024)
    a = gpu_quantize(bits)
    b = gpu_quantize(bits)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def _sampled_rows(rng, rows, n=192):
    return np.unique(np.concatenate([[0, rows - 1], rng.integers(0, rows, n)]))


@pytest.mark.parametrize("name,tensors", [
    ("prefill_7b", ("A", "W1", "W2")), ("rotated", ("A", "W")), ("decode", ("A", "W")),
    ("large", ("A", "W")), ("large", ("Q",))])
def test_workload_full_size(name, tensors):
    """Full-size tensors of each workload quantized on the GPU in the bench's
    launch configuration; s32 checked exactly, codes and scales on sampled rows
    (the oracle quantizes those rows with the full-tensor s32)."""
    log(f"generate {name} {tensors}")
    wl = W.get(name, tensors=tensors)
    rng = np.random.default_rng(5)
    for tname in tensors:
        bits = wl.tensors[tname]
        log(f"{name}.{tname} shape={bits.shape}")
        codes, scales, s = gpu_quantize(bits)
        s_ref = Q.tensor_scale(bits)
        assert host(s)[0] == s_ref
        rows = _sampled_rows(rng, bits.shape[0])
        ref = Q.quantize(bits[rows], s32=s_ref)
        idx = torch.from_numpy(rows).to("cuda")
        np.testing.assert_array_equal(host(scales.index_select(0, idx)), ref.scales)
        np.testing.assert_array_equal(host(codes.index_select(0, idx)), ref.codes)
        log(f"{name}.{tname} ok; E1M2 share {ref.t.mean():.3f}")


@pytest.mark.parametrize("tie_share", [1.0, 0.5])
def test_many_undecided_blocks(tie_share):
    """Blocks with one nonzero element +-42 * 2^e: E2M1 under the scale 7 * 2^e
    and INT4 under 6 * 2^e both hold it exactly, so the two errors tie and only
    the exact decision settles the block (T = 1).  A 6144 x 4096 tensor of
    them (half of them among random blocks at tie_share 0.5): every wave of
    the streaming quantizer takes its exact path, many times over.  s32 given
    (1) and computed (672 / 2688 = 1/4 keeps the ties); codes and scales on
    sampled rows."""
    rng = np.random.default_rng(11)
    rows, k = 6144, 4096
    nb = rows * k // 16
    x = np.zeros((nb, 16), np.float32)
    tie = rng.random(nb) < tie_share
    val = 42.0 * np.exp2(rng.integers(-4, 5, nb)) * np.where(rng.random(nb) < 0.5, -1.0, 1.0)
    x[np.arange(nb), rng.integers(0, 16, nb)] = np.where(tie, val, 0.0)
    x[~tie] = rng.standard_normal((int((~tie).sum()), 16)) * 3.0
    tie[0] = True                                   # block 0 holds the tensor maximum
    x[0] = 0.0
    x[0, 0] = 672.0                                 # 42 * 16; s32 = 672 / 2688 = 1/4
    bits = W.f32_to_bf16_bits(x.reshape(rows, k))
    for s32 in (1.0, None):
        log(f"undecided blocks tie_share={tie_share} s32={s32}")
        codes, scales, s = gpu_quantize(bits, s32)
        s_ref = np.float32(s32) if s32 is not None else Q.tensor_scale(bits)
        assert s_ref == np.float32(1.0 if s32 is not None else 0.25)
        assert host(s)[0] == s_ref
        sample = _sampled_rows(rng, rows, 48)
        ref = Q.quantize(bits[sample], s32=s_ref)
        idx = torch.from_numpy(sample).to("cuda")
        np.testing.assert_array_equal(host(scales.index_select(0, idx)), ref.scales)
        np.testing.assert_array_equal(host(codes.index_select(0, idx)), ref.codes)
        assert (ref.delta[tie.reshape(rows, k // 16)[sample]] == 0).all()


def test_four_six_ties_and_full_size():
    """4/6 on blocks where both candidates are exact (ties keep max/6), and
    on the full 7B-class prefill activation (sampled rows)."""
    import paper_2605_31035_amd as M
    x = np.zeros((2, 32), np.float32)
    x[0, 0] = 6.0
    x[0, 16:18] = [3.0, -1.5]
    x[1, :16] = np.arange(16) * 0.25
    bits = W.f32_to_bf16_bits(x)
    codes, scales, _ = M.mixfp4_quantize(dev_bf16(bits), dev_f32(1.0), mode="four_six")
    torch.cuda.synchronize()
    ref = Q.quantize(bits, s32=1.0, mode="four_six")
    np.testing.assert_array_equal(host(scales), ref.scales)
    np.testing.assert_array_equal(host(codes), ref.codes)
    assert host(scales)[0, 0] == 0x38 and host(scales)[0, 1] == 0x30
    a = W.get("prefill_7b", tensors=("A",)).tensors["A"]
    log("four_six full size prefill A")
    codes, scales, s = M.mixfp4_quantize(dev_bf16(a), mode="four_six")
    torch.cuda.synchronize()
    s32 = Q.tensor_scale(a)
    assert host(s)[0] == s32
    rows = np.unique(np.random.default_rng(3).integers(0, a.shape[0], 64))
    ref = Q.quantize(a[rows], s32=s32, mode="four_six")
    np.testing.assert_array_equal(host(scales)[rows], ref.scales)
    np.testing.assert_array_equal(host(codes)[rows], ref.codes)
