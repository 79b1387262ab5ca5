"""CPU checks of the C ABI: the library loads, exports every function that
include/mixfp4.h declares, and rejects bad arguments on the host before
anything reaches a GPU (no kernel is launched by these calls)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mixfp4.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mixfp4_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2605_31035_amd import _lib
    return _lib.lib


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert {"mixfp4_quantize", "mixfp4_dequantize", "mixfp4_gemm"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name
    from paper_2605_31035_amd import _lib
    assert set(_lib.SYMBOLS) == set(names)


def test_abi_version(lib):
    v = re.search(r"#define MIXFP4_ABI_VERSION (\d+)", open(HEADER).read()).group(1)
    assert lib.mixfp4_abi_version() == int(v)


def test_status_strings(lib):
    for st, key in [(0, b"OK"), (1, b"NULL"), (2, b"SHAPE"), (3, b"ALIGN"), (4, b"FLAGS"), (5, b"LAUNCH")]:
        assert key in lib.mixfp4_status_string(st)
    assert b"unknown" in lib.mixfp4_status_string(99)


P = ctypes.c_void_p
A16 = P(0x10000)          # a fake, 16-byte aligned address: never dereferenced
A4 = P(0x10004)


def q(lib, x=A16, rows=4, k=32, ldx=32, codes=A16, scales=A16, ts=A16, flags=0):
    return lib.mixfp4_quantize(x, rows, k, ldx, codes, scales, ts, flags, None)


def test_quantize_rejects(lib):
    assert q(lib, flags=7) == 4          # both FORCE bits (with GIVEN)
    assert q(lib, flags=6) == 4          # both FORCE bits
    assert q(lib, flags=8) == 4          # STOCHASTIC needs mixfp4_quantize_ex
    assert q(lib, flags=16) == 4         # TRANSPOSE is a mixfp4_quantize_ex option
    assert q(lib, flags=64) == 4         # unknown bit
    assert q(lib, flags=2 | 32) == 4     # two format modes
    assert q(lib, flags=4 | 32) == 4
    assert q(lib, flags=0x80000002) == 4
    assert q(lib, k=24) == 2
    assert q(lib, k=-16) == 2
    assert q(lib, rows=-1) == 2
    assert q(lib, ldx=16) == 2            # ldx < k
    assert q(lib, ldx=36) == 2            # ldx % 8
    assert q(lib, ts=P(0)) == 1
    assert q(lib, x=P(0)) == 1
    assert q(lib, codes=P(0)) == 1
    assert q(lib, scales=P(0)) == 1
    assert q(lib, x=P(0x10008)) == 3
    assert q(lib, codes=P(0x10008)) == 3
    assert q(lib, ts=P(0x10002)) == 3


def test_dequantize_rejects(lib):
    f = lib.mixfp4_dequantize
    assert f(A16, A16, None, 2, 20, A16, None) == 2
    assert f(A16, A16, None, -2, 32, A16, None) == 2
    assert f(P(0), A16, None, 2, 32, A16, None) == 1
    assert f(A16, A16, None, 2, 32, P(0), None) == 1
    assert f(P(0x10008), A16, None, 2, 32, A16, None) == 3
    assert f(A16, A16, None, 2, 32, A4, None) == 3
    assert f(A16, A16, P(0x10001), 2, 32, A16, None) == 3
    assert f(P(0), P(0), None, 0, 32, P(0), None) == 0      # empty: nothing to do


def test_gemm_rejects(lib):
    f = lib.mixfp4_gemm
    args = lambda **kw: [kw.get(n, d) for n, d in [
        ("ac", A16), ("asc", A16), ("ats", None), ("wc", A16), ("wsc", A16), ("wts", None),
        ("m", 8), ("n", 8), ("k", 32), ("c", A16), ("s", None)]]
    assert f(*args(k=40)) == 2
    assert f(*args(m=-1)) == 2
    assert f(*args(c=P(0))) == 1
    assert f(*args(ac=P(0))) == 1
    assert f(*args(wsc=P(0))) == 1
    assert f(*args(ac=P(0x10008))) == 3
    assert f(*args(c=P(0x10002))) == 3
    assert f(*args(ats=P(0x10002))) == 3
    assert f(*args(m=0, ac=P(0), c=P(0))) == 0                # empty output: no-op


def qx(lib, x=A16, rows=4, k=256, ldx=256, codes=A16, scales=A16, ts=A16, flags=0, block=0,
       signs=None, seed=0, offset=0):
    return lib.mixfp4_quantize_ex(x, rows, k, ldx, codes, scales, ts, flags, block, signs, seed,
                                  offset, None)


def test_quantize_ex_rejects(lib):
    assert qx(lib, flags=64) == 4
    assert qx(lib, flags=2 | 32) == 4
    assert qx(lib, flags=6 | 8) == 4
    assert qx(lib, flags=16, rows=4) == 2                # transpose: rows % 16
    assert qx(lib, flags=16, rows=256, block=128) == 2   # transposed rotation: b <= 64
    assert qx(lib, flags=16, rows=48, block=32) == 2     # rows % b
    for bad in (8, 48, 512, -16, 1):
        assert qx(lib, block=bad) == 2, bad
    assert qx(lib, k=96, ldx=96, block=64) == 2       # block does not divide k
    assert qx(lib, k=24, ldx=24) == 2
    assert qx(lib, x=P(0), block=16) == 1
    assert qx(lib, ts=P(0), flags=8) == 1
    assert qx(lib, codes=P(0x10008), block=128) == 3
    # empty input in GIVEN mode: nothing to launch, success
    assert qx(lib, rows=0, flags=1 | 8, block=256) == 0


def test_hadamard_rejects(lib):
    f = lib.mixfp4_hadamard
    for bad in (0, 8, 24, 512):
        assert f(A16, 2, 256, 256, bad, None, A16, None) == 2, bad
    assert f(A16, 2, 96, 96, 64, None, A16, None) == 2
    assert f(A16, 2, 128, 120, 16, None, A16, None) == 2   # ldx < k
    assert f(A16, 2, 128, 132, 16, None, A16, None) == 2   # ldx % 8
    assert f(P(0), 2, 128, 128, 16, None, A16, None) == 1
    assert f(A16, 2, 128, 128, 16, None, P(0), None) == 1
    assert f(A16, 2, 128, 128, 16, None, P(0x10008), None) == 3
    assert f(A16, 0, 128, 128, 16, None, P(0), None) == 0     # empty: nothing to do


def test_quantize_2d_rejects(lib):
    def f(w=A16, rows=32, k=64, ldw=64, codes=A16, scales=A16, ct=A16, st=A16, ts=A16, flags=0):
        return lib.mixfp4_quantize_2d(w, rows, k, ldw, codes, scales, ct, st, ts, flags, None)
    assert f(flags=8) == 4
    assert f(flags=6) == 4
    assert f(flags=36) == 4
    assert f(rows=24) == 2
    assert f(k=40, ldw=40) == 2
    assert f(ldw=60) == 2
    assert f(ts=P(0)) == 1
    assert f(ct=P(0)) == 1                 # codes_t and scales_t go together
    assert f(codes=P(0)) == 1
    assert f(ct=P(0x10008)) == 3
    assert f(rows=0, flags=1) == 0


# --- the Python binding rejects mis-shaped tensors before any launch --------
# (CPU tensors: every check below fires before the device check, and a
# correctly shaped CPU argument is rejected for its device, so no call reaches
# the library.)

def _gemm_args(m=32, n=48, k=64):
    import torch
    u8 = torch.uint8
    a = (torch.zeros((m, k // 2), dtype=u8), torch.zeros((m, k // 16), dtype=u8),
         torch.ones(1, dtype=torch.float32))
    w = (torch.zeros((n, k // 2), dtype=u8), torch.zeros((n, k // 16), dtype=u8),
         torch.ones(1, dtype=torch.float32))
    return a, w, torch.zeros((m, n), dtype=torch.float32)


def test_binding_gemm_rejects_bad_tensors():
    import torch

    import paper_2605_31035_amd as M
    a, w, out = _gemm_args()
    cases = [
        ((a, w, out[:, :40]), "out must have shape"),                       # short out
        ((a, w, out.t().contiguous().t()), "contiguous"),                   # strided out
        ((a, w, out.double()), "float32"),                                  # wrong dtype
        (((a[0], a[1][:, :3], a[2]), w, out), "A scales must have shape"),  # scales too narrow
        (((a[0][:, :16], a[1], a[2]), w, None), "disagree on K"),           # K-sliced codes
        (((a[0][:, ::2], a[1][:, :2], a[2]), (w[0][:, :16], w[1][:, :2], w[2]), None),
         "contiguous"),                                                     # strided codes
        ((a, (w[0], w[1].to(torch.int8), w[2]), out), "uint8"),
        (((a[0], a[1], torch.ones(2)), w, out), "1 element"),
        ((a, w, out), "CUDA tensor"),                                       # all fine but CPU
    ]
    for (aa, ww, oo), msg in cases:
        with pytest.raises(ValueError, match=msg):
            M.mixfp4_gemm(aa, ww, out=oo)


def test_binding_dequantize_rejects_bad_tensors():
    import torch

    import paper_2605_31035_amd as M
    codes = torch.zeros((4, 32), dtype=torch.uint8)
    scales = torch.zeros((4, 4), dtype=torch.uint8)
    with pytest.raises(ValueError, match="scales must have shape"):
        M.mixfp4_dequantize(codes, scales[:, :3])
    with pytest.raises(ValueError, match="contiguous"):
        M.mixfp4_dequantize(torch.zeros((4, 64), dtype=torch.uint8)[:, ::2], scales)
    with pytest.raises(ValueError, match="multiple of 16"):
        M.mixfp4_dequantize(torch.zeros((4, 4), dtype=torch.uint8), scales[:, :0])
    with pytest.raises(ValueError, match="1 element"):
        M.mixfp4_dequantize(codes, scales, torch.ones(3))
    with pytest.raises(ValueError, match="CUDA tensor"):
        M.mixfp4_dequantize(codes, scales)


def test_binding_quantize_rejects_bad_outputs():
    import torch

    import paper_2605_31035_amd as M
    x = torch.zeros((8, 64), dtype=torch.bfloat16)
    good_c = torch.zeros((8, 32), dtype=torch.uint8)
    good_s = torch.zeros((8, 4), dtype=torch.uint8)
    with pytest.raises(ValueError, match="codes must have shape"):
        M.mixfp4_quantize(x, codes=good_c[:, :16].contiguous(), scales=good_s)
    with pytest.raises(ValueError, match="scales must have shape"):
        M.mixfp4_quantize(x, codes=good_c, scales=good_s[:4])
    with pytest.raises(ValueError, match="scale_out must have 1 element"):
        M.mixfp4_quantize(x, codes=good_c, scales=good_s, scale_out=torch.ones(2))
    with pytest.raises(ValueError, match="codes must have shape"):
        M.mixfp4_quantize(x, codes=good_c, scales=good_s, transpose=True)
    with pytest.raises(ValueError, match="CUDA tensor"):
        M.mixfp4_quantize(x, codes=good_c, scales=good_s)


def test_gemm_ws_rejects(lib):
    f = lib.mixfp4_gemm_ws
    args = lambda **kw: [kw.get("ac", A16), kw.get("as_", A16), None, kw.get("wc", A16),
                         kw.get("ws", A16), None, kw.get("m", 64), kw.get("n", 64),
                         kw.get("k", 64), kw.get("c", A16), kw.get("work", P(0x10000)),
                         kw.get("wb", 1 << 20), None]
    assert f(*args(k=24)) == 2                      # k % 16
    assert f(*args(m=-1)) == 2
    assert f(*args(wb=-1)) == 2                     # negative workspace size
    assert f(*args(c=None)) == 1
    assert f(*args(ac=None)) == 1
    assert f(*args(work=P(0x10080))) == 3           # workspace not 256-byte aligned
    assert f(*args(c=P(0x10002))) == 3
    assert f(*args(m=0)) == 0                       # nothing to compute, nothing launched


def test_gemm_workspace_size(lib):
    b = ctypes.c_int64(-1)
    assert lib.mixfp4_gemm_workspace_size(16384, 8192, 8192, ctypes.byref(b)) == 0
    assert b.value == (16384 + 8192) * 8192 * 2
    assert lib.mixfp4_gemm_workspace_size(300, 1000, 288, ctypes.byref(b)) == 0
    assert b.value == (512 + 1024) * 288 * 2
    assert lib.mixfp4_gemm_workspace_size(16, 4096, 4096, ctypes.byref(b)) == 0 and b.value == 0
    assert lib.mixfp4_gemm_workspace_size(64, 64, 48, ctypes.byref(b)) == 0 and b.value == 0
    assert lib.mixfp4_gemm_workspace_size(64, 64, 40, ctypes.byref(b)) == 2
    assert lib.mixfp4_gemm_workspace_size(64, 64, 64, None) == 1


def test_decode_operand_and_decoded_gemm_reject(lib):
    need = ctypes.c_int64(-1)
    assert lib.mixfp4_decode_operand(None, None, 300, 288, None, 0, ctypes.byref(need), None) == 0
    assert need.value == 512 * 288 * 2
    assert lib.mixfp4_decode_operand(A16, A16, 300, 48, A16, 1 << 30, None, None) == 2   # k % 32
    assert lib.mixfp4_decode_operand(A16, A16, -1, 64, A16, 1 << 30, None, None) == 2
    assert lib.mixfp4_decode_operand(A16, A16, 300, 288, P(0x10000), 1000, None, None) == 2  # short
    assert lib.mixfp4_decode_operand(A16, A16, 300, 288, P(0x10010), 1 << 30, None, None) == 3
    assert lib.mixfp4_decode_operand(None, A16, 300, 288, P(0x10000), 1 << 30, None, None) == 1
    g = lib.mixfp4_gemm_decoded
    assert g(P(0x10000), None, P(0x10000), None, 64, 64, 48, A16, None) == 2
    assert g(P(0x10000), None, P(0x10040), None, 64, 64, 64, A16, None) == 3
    assert g(P(0x10000), None, None, None, 64, 64, 64, A16, None) == 1
    assert g(P(0x10000), None, P(0x10000), None, 0, 64, 64, None, None) == 0


def test_two_pass_rule():
    """The binding's path rule (host logic only): two passes for the large and
    rotated GEMM shapes, the fused kernel for the 2048-row prefill shapes, and
    never where the two-pass path does not apply."""
    import paper_2605_31035_amd as M
    assert M.gemm_two_pass_preferred(16384, 8192, 8192)
    assert M.gemm_two_pass_preferred(4096, 14336, 4096)
    assert M.gemm_two_pass_preferred(4096, 4096, 4096)          # m n / (m + n) = 2048 exactly
    assert M.gemm_two_pass_preferred(2048, 11008, 4096)
    assert M.gemm_two_pass_preferred(2048, 4096, 4096)
    assert not M.gemm_two_pass_preferred(1024, 4096, 4096)
    assert not M.gemm_two_pass_preferred(16, 1 << 20, 4096)     # decode shape: fused
    assert not M.gemm_two_pass_preferred(16384, 16384, 48)      # k % 32 != 0


def test_decode_step_rejects(lib):
    """mixfp4_decode_step's argument checks, all before any device access."""
    f = lib.mixfp4_decode_step
    args = lambda **kw: [kw.get("a", A16), kw.get("m", 16), kw.get("k", 4096), A16, A16, None,
                         kw.get("n", 64), kw.get("ac", A16), kw.get("as_", A16), A16,
                         kw.get("c", A16), kw.get("sync", A16), None]
    assert f(*args(a=None)) == 1
    assert f(*args(sync=None)) == 1
    assert f(*args(c=None)) == 1
    assert f(*args(m=17)) == 2                      # more than 16 rows
    assert f(*args(m=0)) == 2
    assert f(*args(k=4096 + 32)) == 2               # k % 64
    assert f(*args(k=4096 + 272)) == 2
    assert f(*args(k=48)) == 2
    assert f(*args(n=0)) == 2
    assert f(*args(a=P(0x10008))) == 3              # A not 16-byte aligned
    assert f(*args(ac=P(0x10008))) == 3
    assert f(*args(as_=P(0x10002))) == 3
    assert f(*args(sync=P(0x10002))) == 3


def test_decode_step_applies_rule():
    import paper_2605_31035_amd as M
    assert M.decode_step_applies(16, 8192) and M.decode_step_applies(1, 512)
    assert M.decode_step_applies(16, 11008) and M.decode_step_applies(3, 256)
    assert M.decode_step_applies(16, 640) and M.decode_step_applies(2, 64)   # K tails
    assert not M.decode_step_applies(17, 8192) and not M.decode_step_applies(16, 4128)
    assert not M.decode_step_applies(4, 48)


def test_quantize_variant_rejects(lib):
    """mixfp4_quantize_variant / mixfp4_dequantize_variant argument checks,
    all before any device access."""
    f = lib.mixfp4_quantize_variant

    def qv(**kw):
        return f(kw.get("x", A16), kw.get("rows", 2), kw.get("k", 64), kw.get("ldx", 64),
                 kw.get("block", 32), kw.get("cand", 5), kw.get("codes", A16),
                 kw.get("scales", A16), kw.get("fmt", A16), kw.get("ts", A16),
                 kw.get("flags", 0), None)

    assert qv(block=24) == 2 and qv(block=128) == 2 and qv(block=0) == 2
    assert qv(cand=0) == 4 and qv(cand=8) == 4
    assert qv(flags=2) == 4 and qv(flags=8) == 4
    assert qv(k=48) == 2                            # k % block
    assert qv(rows=-1) == 2 and qv(ldx=32) == 2 and qv(ldx=68) == 2
    assert qv(ts=P(0)) == 1 and qv(x=P(0)) == 1 and qv(codes=P(0)) == 1
    assert qv(scales=P(0)) == 1
    assert qv(cand=7, fmt=P(0)) == 1                # three candidates need the index array
    assert qv(x=P(0x10008)) == 3 and qv(codes=P(0x10008)) == 3 and qv(ts=P(0x10002)) == 3
    d = lib.mixfp4_dequantize_variant
    assert d(A16, A16, A16, None, 2, 64, 24, 5, A16, None) == 2
    assert d(A16, A16, A16, None, 2, 64, 32, 0, A16, None) == 4
    assert d(A16, A16, A16, None, 2, 48, 32, 5, A16, None) == 2
    assert d(A16, A16, P(0), None, 2, 64, 32, 7, A16, None) == 1
    assert d(P(0), A16, A16, None, 2, 64, 32, 5, A16, None) == 1
    assert d(A16, A16, A16, None, 2, 64, 32, 5, A4, None) == 3
    assert d(P(0), P(0), P(0), None, 0, 64, 32, 5, P(0), None) == 0    # empty


def test_binding_variant_rejects():
    import torch

    import paper_2605_31035_amd as M
    x = torch.zeros((2, 64), dtype=torch.bfloat16)
    for kw in (dict(block=24), dict(candidates=()), dict(candidates=("e2m1", "e2m1")),
               dict(candidates=("e4m3",)), dict(block=128)):
        with pytest.raises(ValueError):
            M.mixfp4_quantize_variant(x, **kw)


def test_quantize_decode_rejects(lib):
    f = lib.mixfp4_quantize_decode

    def qd(**kw):
        return f(kw.get("x", A16), kw.get("rows", 2), kw.get("k", 64), kw.get("ldx", 64),
                 kw.get("codes", A16), kw.get("scales", A16), kw.get("ts", A16),
                 kw.get("out", P(0x10000)), kw.get("out_bytes", 1 << 20), kw.get("flags", 0), None)

    assert qd(flags=8) == 4 and qd(flags=6) == 4 and qd(flags=16) == 4
    assert qd(k=48) == 2 and qd(k=1 << 23) == 2 and qd(rows=-1) == 2 and qd(ldx=32) == 2
    assert qd(out_bytes=100) == 2                   # smaller than the decoded layout
    assert qd(ts=P(0)) == 1 and qd(x=P(0)) == 1 and qd(out=P(0)) == 1 and qd(codes=P(0)) == 1
    assert qd(out=P(0x10010)) == 3 and qd(x=P(0x10008)) == 3 and qd(ts=P(0x10002)) == 3
