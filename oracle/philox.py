"""Philox4x32-10 (Salmon, Moraes, Dror, Shaw: "Parallel random numbers: as easy
as 1, 2, 3", SC'11), written from the published description.

One Philox-4x32 round maps the 4-word counter (c0, c1, c2, c3) with the
2-word round key (k0, k1) to
    (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))
with the multipliers M0 = 0xD2511F53, M1 = 0xCD9E8D57; the key is bumped
by the Weyl constants (0x9E3779B9, 0xBB67AE85) between rounds; ten rounds.

Counter assignment used by the draft-and-verify iteration (a reading: the
paper uses greedy decoding and names no generator):
    key = (seed & 0xffffffff, seed >> 32)
    ctr = (sequence b, step & 0xffffffff, step >> 32, (purpose << 16) | index)
    purpose 0 = draft sample at draft slot ``index``
    purpose 1 = accept test of draft position ``index`` (0-based)
    purpose 2 = resample / bonus draw (index 0)
and the 32-bit word drawn is output word 0.
"""
from __future__ import annotations

MASK32 = 0xFFFFFFFF
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85

PURPOSE_DRAFT = 0
PURPOSE_ACCEPT = 1
PURPOSE_RESAMPLE = 2


def philox4x32_10(ctr, key):
    """Return the 4 output words of Philox4x32 with 10 rounds."""
    c0, c1, c2, c3 = (int(x) & MASK32 for x in ctr)
    k0, k1 = (int(x) & MASK32 for x in key)
    for _ in range(10):
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0) & MASK32, p1 & MASK32, \
                         ((p0 >> 32) ^ c3 ^ k1) & MASK32, p0 & MASK32
        k0 = (k0 + PHILOX_W0) & MASK32
        k1 = (k1 + PHILOX_W1) & MASK32
    return c0, c1, c2, c3


def draw_u32(seed: int, b: int, step: int, purpose: int, index: int) -> int:
    """The 32-bit word for (sequence, step, purpose, index) under ``seed``."""
    key = (seed & MASK32, (seed >> 32) & MASK32)
    ctr = (b, step & MASK32, (step >> 32) & MASK32, ((purpose & 0xFFFF) << 16) | (index & 0xFFFF))
    return philox4x32_10(ctr, key)[0]


def uniform_from_u32(x: int):
    """u = (x >> 8) * 2^-24, an exact float32 value in [0, 1)."""
    import numpy as np
    return np.float32((int(x) >> 8) * (2.0 ** -24))
