"""Philox4x32-10 counter-based random numbers, and the per-element uniform
draws of the stochastic-rounding quantizer.

TEST INFRASTRUCTURE (oracle); see ``oracle/__init__``.

Philox4x32-10 is the counter-based generator of Salmon, Moraes, Dror and Shaw,
"Parallel Random Numbers: As Easy as 1, 2, 3" (SC 2011).  Written here from
its published definition:
  * state: a 128-bit counter (four 32-bit words c0..c3) and a 64-bit key
    (k0, k1);
  * one round: with the multipliers M0 = 0xD2511F53 and M1 = 0xCD9E8D57,
    (hi0, lo0) = M0 * c0 and (hi1, lo1) = M1 * c2 as 64-bit products, and the
    new counter is (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0);
  * between rounds the key advances by the Weyl constants
    (k0, k1) += (0x9E3779B9, 0xBB67AE85) mod 2^32;
  * ten rounds; the final counter is the output.
Pinned by the generator's published known-answer vectors.

Draws of the stochastic-rounding quantizer (App. D needs one uniform epsilon
per element): block g of a [rows, K] tensor (g = row * K/16 + column block)
takes Philox4x32-10 with key (seed mod 2^32, seed >> 32) and counter
(g mod 2^32, g >> 32, offset mod 2^32, offset >> 32); element j of the block
gets byte j mod 4 of output word j // 4 (least significant byte first), an
integer u in [0, 256).  The uniform is epsilon = (u + 1/2) / 256.
"""
from __future__ import annotations

import numpy as np

M0 = 0xD2511F53
M1 = 0xCD9E8D57
W0 = 0x9E3779B9
W1 = 0xBB67AE85
ROUNDS = 10
MASK = 0xFFFFFFFF


def philox4x32(counter: np.ndarray, key: np.ndarray, rounds: int = ROUNDS) -> np.ndarray:
    """Philox4x32 of ``counter`` (uint32 [..., 4]) under ``key`` (uint32
    [..., 2], broadcast against the counters); returns uint32 [..., 4]."""
    c = np.asarray(counter, dtype=np.uint64) & MASK
    k = np.broadcast_to(np.asarray(key, dtype=np.uint64) & MASK, c.shape[:-1] + (2,))
    c0, c1, c2, c3 = (c[..., i].copy() for i in range(4))
    k0, k1 = k[..., 0].copy(), k[..., 1].copy()
    for r in range(rounds):
        if r:
            k0 = (k0 + W0) & MASK
            k1 = (k1 + W1) & MASK
        p0 = np.uint64(M0) * c0                 # < 2^64: exact in uint64
        p1 = np.uint64(M1) * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def block_bytes(rows: int, k: int, seed: int, offset: int = 0, row_index=None) -> np.ndarray:
    """The integers u (uint8 [rows, K]) that the stochastic-rounding quantizer
    draws for a [rows, K] tensor under ``seed`` and ``offset`` (64-bit each).
    ``row_index`` (optional) gives the rows' indices in a larger tensor, for
    checking a sample of its rows."""
    assert k % 16 == 0
    nb = k // 16
    r = np.arange(rows, dtype=np.uint64) if row_index is None else np.asarray(row_index, np.uint64)
    assert r.shape == (rows,)
    g = (r[:, None] * np.uint64(nb) + np.arange(nb, dtype=np.uint64)[None, :]).reshape(-1)
    ctr = np.stack([g & MASK, g >> np.uint64(32),
                    np.full_like(g, offset & MASK), np.full_like(g, (offset >> 32) & MASK)], axis=-1)
    key = np.array([seed & MASK, (seed >> 32) & MASK], dtype=np.uint64)
    words = philox4x32(ctr, key)                         # [blocks, 4]
    shifts = np.array([0, 8, 16, 24], dtype=np.uint32)
    u = (words[:, :, None] >> shifts[None, None, :]) & np.uint32(0xFF)   # [blocks, word, byte]
    return u.reshape(rows, k).astype(np.uint8)
