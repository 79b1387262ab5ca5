"""MixFP4 on MI355X: Python binding of libmixfp4.so.

The binding only marshals arguments: torch supplies device memory and the
current HIP stream, every step of the quantizer, dequantizer and GEMM runs in
the library's HIP kernels.  There is no CPU fallback: if the library is
missing or fails to load, importing the low-level handle raises.

Functions (same names as the C ABI in include/mixfp4.h):
  mixfp4_quantize(x, tensor_scale=None, ..., mode="mixfp4", rounding="nearest",
                  seed=0, offset=0, hadamard_block=0, hadamard_signs=None)
      -> (codes, scales, s32)   (the C call is mixfp4_quantize_ex when
                                  rotating or rounding stochastically)
  mixfp4_quantize(..., transpose=True) quantizes X^T (WGRAD operands)
  mixfp4_quantize_2d(w, tensor_scale=None, mode="mixfp4", transposed=True)
      -> (codes, scales, s32) for W and (codes_t, scales_t, s32) for W^T
  mixfp4_hadamard(x, block, signs=None) -> bf16 tensor
  mixfp4_dequantize(codes, scales, tensor_scale=None) -> fp32 tensor
  mixfp4_gemm(a, w, workspace=None) -> C = A W^T (fp32), a/w are (codes, scales,
      s32) triples; with a workspace (a uint8 CUDA tensor, or True to allocate
      one of mixfp4_gemm_workspace_size bytes) the call is mixfp4_gemm_ws
  mixfp4_gemm_workspace_size(m, n, k) -> bytes
  mixfp4_decode_operand((codes, scales, s32)) -> Decoded (the operand decoded
      once to exact 16-bit values in the library's blocked layout)
  mixfp4_gemm_decoded(a: Decoded, w: Decoded) -> C = A W^T (fp32)
"""
from __future__ import annotations

import ctypes
import os
from typing import NamedTuple

import torch

from ._lib import LIB_PATH, MixFP4Error, lib

__all__ = ["mixfp4_decode_step", "decode_step_applies", "gemm_two_pass_preferred", "mixfp4_quantize", "mixfp4_quantize_ex", "mixfp4_hadamard", "mixfp4_dequantize",
           "mixfp4_gemm", "MixFP4Error", "LIB_PATH", "lib", "SCALE_COMPUTE", "SCALE_GIVEN",
           "FORCE_E2M1", "FORCE_E1M2", "STOCHASTIC", "TRANSPOSE", "mixfp4_quantize_2d",
           "mixfp4_gemm_workspace_size", "mixfp4_decode_operand", "mixfp4_gemm_decoded",
           "Decoded", "mixfp4_quantize_variant", "mixfp4_dequantize_variant", "Variant",
           "CANDIDATES", "mixfp4_quantize_decode"]

SCALE_COMPUTE = 0
SCALE_GIVEN = 1
FORCE_E2M1 = 2
FORCE_E1M2 = 4
STOCHASTIC = 8
TRANSPOSE = 16
FOUR_SIX = 32
_MODES = {"mixfp4": 0, "e2m1": FORCE_E2M1, "e1m2": FORCE_E1M2, "four_six": FOUR_SIX}


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _require(t, name: str, dtype, shape=None, numel=None):
    """Check a caller-supplied tensor before its address reaches the library:
    the C ABI takes bare pointers with no pitches, so a wrong dtype, shape or
    layout would make a kernel read or write the wrong bytes.  Shape, dtype
    and contiguity are checked before the device, so every mistake is named."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must have {numel} element(s), got {t.numel()}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _same_device(device, *named):
    """Every tensor on the same CUDA device as the first."""
    for name, t in named:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be a CUDA tensor")
        if t.device != device:
            raise ValueError(f"{name} is on {t.device}, expected {device}")


def _check(status: int):
    if status != 0:
        msg = lib.mixfp4_status_string(status).decode()
        if status == 5:
            msg += ": " + lib.mixfp4_last_launch_error().decode()
        raise MixFP4Error(status, msg)


def mixfp4_quantize(x: torch.Tensor, tensor_scale: torch.Tensor | None = None,
                    codes: torch.Tensor | None = None, scales: torch.Tensor | None = None,
                    scale_out: torch.Tensor | None = None, mode: str = "mixfp4",
                    rounding: str = "nearest", seed: int = 0, offset: int = 0,
                    hadamard_block: int = 0, hadamard_signs: torch.Tensor | None = None,
                    transpose: bool = False):
    """Quantize a bf16 [rows, k] CUDA tensor (Algorithm 1).

    ``tensor_scale`` None computes s32 = max|X| / 2688 on the device (into
    ``scale_out`` if given); a 1-element fp32 tensor is used as the given s32.
    ``mode`` "mixfp4" selects the format per block; "e2m1" (NVFP4) and "e1m2"
    (INT4) take that branch for every block; "four_six" is the 4/6 baseline
    (E2M1 under max/6 or max/4, plain NVFP4 output).  ``rounding`` "stochastic"
    writes the codes by App. D's stochastic rounding with Philox draws of
    (``seed``, ``offset``).  ``hadamard_block`` b > 0 rotates X first
    (mixfp4_hadamard with ``hadamard_signs``, an int8 CUDA tensor of b signs).
    ``transpose`` quantizes X^T instead (blocks of 16 rows of X; a rotation
    then runs along the rows).
    Returns (codes uint8 [rows, k/2], scales uint8 [rows, k/16], s32 fp32 [1]),
    or [k, rows/2] and [k, rows/16] with ``transpose``."""
    if mode not in _MODES:
        raise ValueError(f"mode must be one of {sorted(_MODES)}")
    if rounding not in ("nearest", "stochastic"):
        raise ValueError("rounding must be 'nearest' or 'stochastic'")
    if x.dtype != torch.bfloat16 or x.dim() != 2:
        raise ValueError("x must be a 2-D bfloat16 CUDA tensor")
    if x.stride(1) != 1:
        raise ValueError("x must have unit stride along K")
    rows, k = x.shape
    dev = x.device
    orows, ok = (k, rows) if transpose else (rows, k)
    if codes is None:
        codes = torch.empty((orows, ok // 2), dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty((orows, ok // 16), dtype=torch.uint8, device=dev)
    _require(codes, "codes", torch.uint8, (orows, ok // 2))
    _require(scales, "scales", torch.uint8, (orows, ok // 16))
    if tensor_scale is None:
        ts = scale_out if scale_out is not None else torch.empty(1, dtype=torch.float32, device=dev)
        flags = SCALE_COMPUTE
    else:
        ts = tensor_scale
        flags = SCALE_GIVEN
    _require(ts, "tensor_scale" if tensor_scale is not None else "scale_out", torch.float32,
             numel=1)
    _same_device(dev, ("x", x), ("codes", codes), ("scales", scales), ("tensor scale", ts))
    flags |= _MODES[mode]
    ldx = x.stride(0) if rows > 0 else k
    if rounding == "nearest" and hadamard_block == 0 and not transpose:
        st = lib.mixfp4_quantize(_ptr(x), rows, k, ldx, _ptr(codes), _ptr(scales), _ptr(ts),
                                 flags, _stream(dev))
    else:
        if rounding == "stochastic":
            flags |= STOCHASTIC
        if transpose:
            flags |= TRANSPOSE
        signs = _signs_arg(hadamard_signs, hadamard_block)
        st = lib.mixfp4_quantize_ex(_ptr(x), rows, k, ldx, _ptr(codes), _ptr(scales), _ptr(ts),
                                    flags, hadamard_block, _ptr(signs),
                                    seed & 0xFFFFFFFFFFFFFFFF, offset & 0xFFFFFFFFFFFFFFFF,
                                    _stream(dev))
    _check(st)
    return codes, scales, ts


mixfp4_quantize_ex = mixfp4_quantize


def _signs_arg(signs, block):
    if signs is None:
        return None
    if signs.dtype != torch.int8 or not signs.is_cuda or not signs.is_contiguous() \
            or signs.numel() != block:
        raise ValueError("hadamard signs must be a contiguous int8 CUDA tensor of `block` entries")
    return signs


def mixfp4_quantize_2d(w: torch.Tensor, tensor_scale: torch.Tensor | None = None,
                       mode: str = "mixfp4", transposed: bool = True,
                       scale_out: torch.Tensor | None = None):
    """2D (16 x 16 tile) quantization of a bf16 weight [n, k] (n, k multiples
    of 16).  Returns ((codes, scales, s32) of W, (codes_t, scales_t, s32) of
    W^T or None): mixfp4_gemm(A, W-part) is FPROP, mixfp4_gemm(dY, W^T-part)
    is DGRAD."""
    if mode not in _MODES:
        raise ValueError(f"mode must be one of {sorted(_MODES)}")
    if w.dtype != torch.bfloat16 or w.dim() != 2 or not w.is_cuda or w.stride(1) != 1:
        raise ValueError("w must be a 2-D bfloat16 CUDA tensor with unit stride along K")
    n, k = w.shape
    dev = w.device
    codes = torch.empty((n, k // 2), dtype=torch.uint8, device=dev)
    scales = torch.empty((n, k // 16), dtype=torch.uint8, device=dev)
    codes_t = torch.empty((k, n // 2), dtype=torch.uint8, device=dev) if transposed else None
    scales_t = torch.empty((k, n // 16), dtype=torch.uint8, device=dev) if transposed else None
    if tensor_scale is None:
        ts = scale_out if scale_out is not None else torch.empty(1, dtype=torch.float32, device=dev)
        flags = SCALE_COMPUTE
    else:
        ts, flags = tensor_scale, SCALE_GIVEN
    _require(ts, "tensor scale", torch.float32, numel=1)
    _same_device(dev, ("tensor scale", ts))
    st = lib.mixfp4_quantize_2d(_ptr(w), n, k, w.stride(0) if n > 0 else k, _ptr(codes),
                                _ptr(scales), _ptr(codes_t), _ptr(scales_t), _ptr(ts),
                                flags | _MODES[mode], _stream(dev))
    _check(st)
    return (codes, scales, ts), ((codes_t, scales_t, ts) if transposed else None)


def mixfp4_hadamard(x: torch.Tensor, block: int, signs: torch.Tensor | None = None,
                    out: torch.Tensor | None = None) -> torch.Tensor:
    """Block-diagonal Hadamard transform of a bf16 [rows, k] CUDA tensor along
    k: each block of ``block`` elements times diag(signs) H / sqrt(block),
    rounded once to bf16.  ``signs``: int8 CUDA tensor of ``block`` entries
    (negative = -1) or None."""
    if x.dtype != torch.bfloat16 or x.dim() != 2 or not x.is_cuda or x.stride(1) != 1:
        raise ValueError("x must be a 2-D bfloat16 CUDA tensor with unit stride along K")
    rows, k = x.shape
    if out is None:
        out = torch.empty((rows, k), dtype=torch.bfloat16, device=x.device)
    _require(out, "out", torch.bfloat16, (rows, k))
    _same_device(x.device, ("out", out))
    sg = _signs_arg(signs, block)
    st = lib.mixfp4_hadamard(_ptr(x), rows, k, x.stride(0) if rows > 0 else k, block, _ptr(sg),
                             _ptr(out), _stream(x.device))
    _check(st)
    return out


def mixfp4_dequantize(codes: torch.Tensor, scales: torch.Tensor,
                      tensor_scale: torch.Tensor | None = None) -> torch.Tensor:
    """Decode MixFP4 to fp32 [rows, k]; ``tensor_scale`` None decodes in the
    FP8 domain (s32 = 1)."""
    if not isinstance(codes, torch.Tensor) or codes.dim() != 2:
        raise ValueError("codes must be a 2-D uint8 tensor [rows, k/2]")
    rows, half = codes.shape
    k = half * 2
    _require(codes, "codes", torch.uint8, (rows, half))
    _require(scales, "scales", torch.uint8, (rows, k // 16))
    if k % 16:
        raise ValueError("k = 2 * codes.shape[1] must be a multiple of 16")
    if tensor_scale is not None:
        _require(tensor_scale, "tensor_scale", torch.float32, numel=1)
    _same_device(codes.device, ("codes", codes), ("scales", scales),
                 ("tensor_scale", tensor_scale))
    out = torch.empty((rows, k), dtype=torch.float32, device=codes.device)
    st = lib.mixfp4_dequantize(_ptr(codes), _ptr(scales), _ptr(tensor_scale), rows, k,
                               _ptr(out), _stream(codes.device))
    _check(st)
    return out


# candidate formats of mixfp4_quantize_variant and their bits in the ABI
CANDIDATES = {"e2m1": 1, "e1m2": 2, "e3m0": 4}


class Variant(NamedTuple):
    """Output of mixfp4_quantize_variant."""
    codes: torch.Tensor      # uint8 [rows, k/2]
    scales: torch.Tensor     # uint8 [rows, k/block]
    fmt: torch.Tensor        # uint8 [rows, k/block], chosen candidate index
    s32: torch.Tensor        # fp32 [1]
    block: int
    mask: int


def _cand_mask(candidates) -> int:
    mask = 0
    for c in candidates:
        if c not in CANDIDATES or mask & CANDIDATES[c]:
            raise ValueError(f"candidates must be distinct names among {sorted(CANDIDATES)}")
        mask |= CANDIDATES[c]
    if not mask:
        raise ValueError("at least one candidate format is needed")
    return mask


def mixfp4_quantize_variant(x: torch.Tensor, block: int = 16, candidates=("e2m1", "e1m2"),
                            tensor_scale: torch.Tensor | None = None) -> Variant:
    """Algorithm 1's block-wise selection over another candidate set and
    block size (mixfp4_quantize_variant): ``candidates`` a subset of
    ("e2m1", "e1m2", "e3m0"), taken in that order whatever the order given;
    ``block`` 8, 16, 32 or 64.  ``tensor_scale`` None computes s32."""
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D bfloat16 CUDA tensor with unit stride along K")
    mask = _cand_mask(candidates)
    rows, k = x.shape
    if block not in (8, 16, 32, 64) or k % block:
        raise ValueError("block must be 8, 16, 32 or 64 and divide k")
    dev = x.device
    codes = torch.empty((rows, k // 2), dtype=torch.uint8, device=dev)
    scales = torch.empty((rows, k // block), dtype=torch.uint8, device=dev)
    fmt = torch.empty((rows, k // block), dtype=torch.uint8, device=dev)
    if tensor_scale is None:
        ts, flags = torch.empty(1, dtype=torch.float32, device=dev), SCALE_COMPUTE
    else:
        ts, flags = tensor_scale, SCALE_GIVEN
        _require(ts, "tensor_scale", torch.float32, numel=1)
    _same_device(dev, ("x", x), ("tensor scale", ts))
    _check(lib.mixfp4_quantize_variant(_ptr(x), rows, k, x.stride(0), block, mask, _ptr(codes),
                                       _ptr(scales), _ptr(fmt), _ptr(ts), flags, _stream(dev)))
    return Variant(codes, scales, fmt, ts, block, mask)


def mixfp4_dequantize_variant(q: Variant, use_fmt: bool = True) -> torch.Tensor:
    """Decode a Variant to fp32 [rows, k] (with its s32).  ``use_fmt`` False
    decodes from the scale bytes alone (possible for sets of one or two)."""
    rows, k = q.codes.shape[0], q.codes.shape[1] * 2
    out = torch.empty((rows, k), dtype=torch.float32, device=q.codes.device)
    _check(lib.mixfp4_dequantize_variant(_ptr(q.codes), _ptr(q.scales),
                                         _ptr(q.fmt) if use_fmt else None, _ptr(q.s32), rows, k,
                                         q.block, q.mask, _ptr(out), _stream(q.codes.device)))
    return out


def mixfp4_gemm_workspace_size(m: int, n: int, k: int) -> int:
    """Bytes of workspace with which mixfp4_gemm(..., workspace=...) takes the
    two-pass path (0 where it does not apply)."""
    b = ctypes.c_int64(0)
    _check(lib.mixfp4_gemm_workspace_size(m, n, k, ctypes.byref(b)))
    return b.value


def gemm_two_pass_preferred(m: int, n: int, k: int) -> bool:
    """Whether the two-pass GEMM (both operands decoded once, then the fp16
    GEMM) is expected to beat the fused kernel for C[m, n] = A W^T: the
    decode costs (m + n) k elements of HBM traffic, the faster GEMM saves a
    share of 2 m n k flops, so it pays off from m n / (m + n) on.  Measured
    on MI355X (decode of W included): 16384x8192x8192 1626 against 1990 us,
    4096x14336x4096 408 against 470 us, 2048x11008x4096 (m n / (m + n) =
    1727) 189 against 219 us and 2048x4096x4096 (1365, on 128 x 256 tiles)
    74 against 89 us favour two passes; smaller products favour the fused
    kernel.  Threshold: 1280."""
    m, n, k = int(m), int(n), int(k)
    return mixfp4_gemm_workspace_size(m, n, k) > 0 and m * n >= 1280 * (m + n)


def mixfp4_gemm(a, w, out: torch.Tensor | None = None, workspace=None) -> torch.Tensor:
    """C = A W^T for MixFP4 operands given as (codes, scales, s32) triples
    (s32 may be None for 1.0).  Returns fp32 [m, n].  ``workspace``: None
    (mixfp4_gemm), a contiguous uint8 CUDA tensor (mixfp4_gemm_ws with it),
    True (mixfp4_gemm_ws with a workspace of mixfp4_gemm_workspace_size bytes
    allocated here), or "auto" (as True where gemm_two_pass_preferred, else
    as None)."""
    ac, asc, ats = a
    wc, wsc, wts = w
    for name, t in (("A codes", ac), ("W codes", wc)):
        if not isinstance(t, torch.Tensor) or t.dim() != 2:
            raise ValueError(f"{name} must be a 2-D uint8 tensor [rows, k/2]")
    m, n, k = ac.shape[0], wc.shape[0], ac.shape[1] * 2
    if wc.shape[1] * 2 != k:
        raise ValueError("A and W disagree on K")
    if k % 16:
        raise ValueError("k = 2 * codes.shape[1] must be a multiple of 16")
    _require(ac, "A codes", torch.uint8, (m, k // 2))
    _require(asc, "A scales", torch.uint8, (m, k // 16))
    _require(wc, "W codes", torch.uint8, (n, k // 2))
    _require(wsc, "W scales", torch.uint8, (n, k // 16))
    for name, t in (("A tensor scale", ats), ("W tensor scale", wts)):
        if t is not None:
            _require(t, name, torch.float32, numel=1)
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=ac.device)
    _require(out, "out", torch.float32, (m, n))
    if isinstance(workspace, str):
        if workspace != "auto":
            raise ValueError('workspace must be None, True, "auto" or a uint8 tensor')
        workspace = True if gemm_two_pass_preferred(m, n, k) else None
    if workspace is True:
        workspace = torch.empty(max(1, mixfp4_gemm_workspace_size(m, n, k)), dtype=torch.uint8,
                                device=ac.device)
    if workspace is not None:
        if not isinstance(workspace, torch.Tensor) or workspace.dtype != torch.uint8 \
                or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous uint8 tensor (or True / None)")
    _same_device(ac.device, ("A codes", ac), ("A scales", asc), ("A tensor scale", ats),
                 ("W codes", wc), ("W scales", wsc), ("W tensor scale", wts), ("out", out),
                 ("workspace", workspace))
    if workspace is None:
        st = lib.mixfp4_gemm(_ptr(ac), _ptr(asc), _ptr(ats), _ptr(wc), _ptr(wsc), _ptr(wts),
                             m, n, k, _ptr(out), _stream(ac.device))
    else:
        st = lib.mixfp4_gemm_ws(_ptr(ac), _ptr(asc), _ptr(ats), _ptr(wc), _ptr(wsc), _ptr(wts),
                                m, n, k, _ptr(out), _ptr(workspace), workspace.numel(),
                                _stream(ac.device))
    _check(st)
    return out


_STEP_SYNC: dict = {}


def decode_step_applies(m: int, k: int) -> bool:
    """Shapes mixfp4_decode_step takes: 1 <= m <= 16 rows, k % 64 == 0."""
    return 1 <= m <= 16 and k > 0 and k % 64 == 0


def mixfp4_decode_step(x: torch.Tensor, w, out: torch.Tensor | None = None, a_out=None,
                       sync: torch.Tensor | None = None):
    """One decode step in one launch (mixfp4_decode_step): quantize the bf16
    activation x [m <= 16, k] (tensor scale computed on the device) and
    return (C = x_q W^T fp32 [m, n], (codes, scales, s32) of x).  ``w`` is a
    quantized (codes, scales, s32) triple.  ``a_out``: optional (codes,
    scales, s32) tensors to write A's outputs into.  ``sync``: 4 zeroed
    int32 on the device that the launch leaves zeroed; default, one per
    device kept by this module (calls on one device must then be ordered,
    e.g. on one stream)."""
    if not isinstance(x, torch.Tensor) or x.dim() != 2 or x.dtype != torch.bfloat16:
        raise ValueError("x must be a 2-D bfloat16 tensor")
    wc, wsc, wts = w
    m, k = x.shape
    n = wc.shape[0] if isinstance(wc, torch.Tensor) and wc.dim() == 2 else -1
    if not decode_step_applies(m, k) or n < 1:
        raise ValueError(f"decode step needs 1 <= m <= 16, k % 64 == 0, n >= 1 (m={m}, k={k}, n={n})")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    _require(wc, "W codes", torch.uint8, (n, k // 2))
    _require(wsc, "W scales", torch.uint8, (n, k // 16))
    if wts is not None:
        _require(wts, "W tensor scale", torch.float32, numel=1)
    dev = x.device
    if a_out is None:
        a_out = (torch.empty((m, k // 2), dtype=torch.uint8, device=dev),
                 torch.empty((m, k // 16), dtype=torch.uint8, device=dev),
                 torch.empty(1, dtype=torch.float32, device=dev))
    ac, asc, ats = a_out
    _require(ac, "A codes", torch.uint8, (m, k // 2))
    _require(asc, "A scales", torch.uint8, (m, k // 16))
    _require(ats, "A tensor scale", torch.float32, numel=1)
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (m, n))
    if sync is None:
        key = (dev.type, dev.index if dev.index is not None else torch.cuda.current_device())
        sync = _STEP_SYNC.get(key)
        if sync is None:
            sync = torch.zeros(4, dtype=torch.int32, device=dev)
            _STEP_SYNC[key] = sync
    _require(sync, "sync", torch.int32, numel=4)
    _same_device(dev, ("x", x), ("W codes", wc), ("W scales", wsc), ("W tensor scale", wts),
                 ("A codes", ac), ("A scales", asc), ("A tensor scale", ats), ("out", out),
                 ("sync", sync))
    _check(lib.mixfp4_decode_step(_ptr(x), m, k, _ptr(wc), _ptr(wsc), _ptr(wts), n, _ptr(ac),
                                  _ptr(asc), _ptr(ats), _ptr(out), _ptr(sync), _stream(dev)))
    return out, (ac, asc, ats)


class Decoded(NamedTuple):
    """An operand decoded by mixfp4_decode_operand: ``buf`` (uint8 CUDA
    tensor in the library's blocked layout), its logical shape and its tensor
    scale (fp32 [1] tensor or None)."""
    buf: torch.Tensor
    rows: int
    k: int
    s32: torch.Tensor | None


def mixfp4_quantize_decode(x: torch.Tensor, tensor_scale: torch.Tensor | None = None,
                           mode: str = "mixfp4", out: torch.Tensor | None = None,
                           codes: torch.Tensor | None = None, scales: torch.Tensor | None = None,
                           scale_out: torch.Tensor | None = None):
    """Quantize a bf16 [rows, k] activation (Algorithm 1, as mixfp4_quantize)
    and decode it for mixfp4_gemm_decoded in the same pass
    (mixfp4_quantize_decode).  ``tensor_scale`` None computes s32 (into
    ``scale_out`` if given).  Returns ((codes, scales, s32), Decoded)."""
    if mode not in _MODES:
        raise ValueError(f"mode must be one of {sorted(_MODES)}")
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D bfloat16 CUDA tensor with unit stride along K")
    rows, k = x.shape
    if k % 32:
        raise ValueError("k must be a multiple of 32 for the decoded GEMM")
    dev = x.device
    need = ctypes.c_int64(0)
    _check(lib.mixfp4_decode_operand(None, None, rows, k, None, 0, ctypes.byref(need), None))
    if out is None:
        out = torch.empty(max(1, need.value), dtype=torch.uint8, device=dev)
    if codes is None:
        codes = torch.empty((rows, k // 2), dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty((rows, k // 16), dtype=torch.uint8, device=dev)
    _require(out, "out", torch.uint8)
    _require(codes, "codes", torch.uint8, (rows, k // 2))
    _require(scales, "scales", torch.uint8, (rows, k // 16))
    if out.numel() < need.value:
        raise ValueError(f"out must hold {need.value} bytes")
    if tensor_scale is None:
        ts = scale_out if scale_out is not None else torch.empty(1, dtype=torch.float32, device=dev)
        flags = SCALE_COMPUTE
    else:
        ts, flags = tensor_scale, SCALE_GIVEN
    _require(ts, "tensor_scale", torch.float32, numel=1)
    _same_device(dev, ("x", x), ("codes", codes), ("scales", scales), ("tensor scale", ts),
                 ("out", out))
    _check(lib.mixfp4_quantize_decode(_ptr(x), rows, k, x.stride(0), _ptr(codes), _ptr(scales),
                                      _ptr(ts), _ptr(out), out.numel(), flags | _MODES[mode],
                                      _stream(dev)))
    return (codes, scales, ts), Decoded(out, rows, k, ts)


def mixfp4_decode_operand(q, out: torch.Tensor | None = None) -> Decoded:
    """Decode a MixFP4 operand (codes [rows, k/2], scales [rows, k/16], s32)
    once into exact 16-bit values (App. B.5) for mixfp4_gemm_decoded; k % 32
    must be 0."""
    codes, scales, ts = q
    if not isinstance(codes, torch.Tensor) or codes.dim() != 2:
        raise ValueError("codes must be a 2-D uint8 tensor [rows, k/2]")
    rows, k = codes.shape[0], codes.shape[1] * 2
    if k % 32:
        raise ValueError("k must be a multiple of 32 for the decoded GEMM")
    _require(codes, "codes", torch.uint8, (rows, k // 2))
    _require(scales, "scales", torch.uint8, (rows, k // 16))
    if ts is not None:
        _require(ts, "tensor scale", torch.float32, numel=1)
    need = ctypes.c_int64(0)
    _check(lib.mixfp4_decode_operand(None, None, rows, k, None, 0, ctypes.byref(need), None))
    if out is None:
        out = torch.empty(max(1, need.value), dtype=torch.uint8, device=codes.device)
    _require(out, "out", torch.uint8)
    if out.numel() < need.value:
        raise ValueError(f"out must hold {need.value} bytes")
    _same_device(codes.device, ("codes", codes), ("scales", scales), ("tensor scale", ts),
                 ("out", out))
    _check(lib.mixfp4_decode_operand(_ptr(codes), _ptr(scales), rows, k, _ptr(out), out.numel(),
                                     None, _stream(codes.device)))
    return Decoded(out, rows, k, ts)


def mixfp4_gemm_decoded(a: Decoded, w: Decoded, out: torch.Tensor | None = None) -> torch.Tensor:
    """C = s32_A s32_W A W^T (fp32 [m, n]) from two decoded operands."""
    if a.k != w.k:
        raise ValueError("A and W disagree on K")
    m, n = a.rows, w.rows
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=a.buf.device)
    _require(out, "out", torch.float32, (m, n))
    _same_device(a.buf.device, ("A", a.buf), ("W", w.buf), ("A tensor scale", a.s32),
                 ("W tensor scale", w.s32), ("out", out))
    _check(lib.mixfp4_gemm_decoded(_ptr(a.buf), _ptr(a.s32), _ptr(w.buf), _ptr(w.s32), m, n, a.k,
                                   _ptr(out), _stream(a.buf.device)))
    return out
