"""GEMM of two MixFP4 operands on the CPU.

TEST INFRASTRUCTURE (oracle); see ``oracle/__init__``.

App. B.1, eq. (factor): a block-scaled operand is A_q (.) s_A with the scale
constant over V = 16 values along the reduction dimension; the product of two
such operands is the ordinary matrix product of the dequantized values.  This
oracle is that definition: both operands are dequantized exactly
(s32 * s8 * v in float64, no rounding) and multiplied with a float64 matmul.

Acceptance bound for a computed C (fp32 accumulation on the GPU):
    |C - C_ref| <= 1e-5 * sum_k |A_hat[m,k] * W_hat[n,k]| + 1e-6.
"""
from __future__ import annotations

import numpy as np

from .quant import dequantize_exact

RTOL = 1e-5
ATOL = 1e-6


def operands(a_q, w_q):
    """Exactly dequantized float64 operands A_hat [M,K], W_hat [N,K]."""
    a = dequantize_exact(a_q.codes, a_q.scales, a_q.s32)
    w = dequantize_exact(w_q.codes, w_q.scales, w_q.s32)
    return a, w


def gemm(a_hat: np.ndarray, w_hat: np.ndarray):
    """C_ref = A_hat W_hat^T and bound = |A_hat| |W_hat|^T, both float64."""
    c = a_hat @ w_hat.T
    bound = np.abs(a_hat) @ np.abs(w_hat).T
    return c, bound


def within_tolerance(c: np.ndarray, c_ref: np.ndarray, bound: np.ndarray):
    """Boolean mask of elements meeting the acceptance bound, and the worst
    ratio |err| / allowed."""
    err = np.abs(c.astype(np.float64) - c_ref)
    allowed = RTOL * bound + ATOL
    return err <= allowed, float(np.max(err / allowed)) if err.size else 0.0
