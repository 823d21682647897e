"""Philox4x32-10, written from its published definition.

Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
SC'11, Sec. 3.3 / Fig. 2: a 4x32-bit counter and a 2x32-bit key; each of the
ten rounds multiplies counter words 0 and 2 by the constants M0 and M1 (full
32x32 -> 64-bit products), then

    c0' = hi(M1*c2) ^ c1 ^ k0,   c1' = lo(M1*c2),
    c2' = hi(M0*c0) ^ c3 ^ k1,   c3' = lo(M0*c0),

and the key is bumped by the Weyl constants (W0, W1) between rounds.

Pure Python integers; slow and obviously exact.  Oracle only (test
infrastructure).
"""
from __future__ import annotations

MASK32 = 0xFFFFFFFF
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85


def philox4x32(ctr, key, rounds: int = 10):
    c0, c1, c2, c3 = (int(v) & MASK32 for v in ctr)
    k0, k1 = (int(v) & MASK32 for v in key)
    for rnd in range(rounds):
        if rnd > 0:
            k0 = (k0 + PHILOX_W0) & MASK32
            k1 = (k1 + PHILOX_W1) & MASK32
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        hi0, lo0 = p0 >> 32, p0 & MASK32
        hi1, lo1 = p1 >> 32, p1 & MASK32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0) & MASK32, lo1, (hi0 ^ c3 ^ k1) & MASK32, lo0
    return (c0, c1, c2, c3)


def cutoff_word(r: int, seed: int, offset: int) -> int:
    """The 32-bit uniform integer x_r that decides completion r's cutoff.

    Counter = (r, 0, low 32 bits of offset, high 32 bits of offset);
    key = (low 32 bits of seed, high 32 bits of seed); word 0 of the output.
    """
    ctr = (r & MASK32, 0, offset & MASK32, (offset >> 32) & MASK32)
    key = (seed & MASK32, (seed >> 32) & MASK32)
    return philox4x32(ctr, key)[0]
