"""Philox4x32-10 (Salmon, Moraes, Dror, Shaw: "Parallel Random Numbers: As Easy
as 1, 2, 3", SC'11), plain Python integers.

One round maps counter (c0, c1, c2, c3) and key (k0, k1) to
  (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))
with M0 = 0xD2511F53, M1 = 0xCD9E8D57; between rounds the key is bumped by the
Weyl constants (0x9E3779B9, 0xBB67AE85).  Ten rounds.

Uniforms: u = ((x >> 9) + 0.5) * 2^-23, which lies in (0, 1) and is exact in
fp32 (at most 24 significant bits; the 24-bit variant would need 25).  Gumbel noise: g = -log(-log u).

Parity: pinned by the generator's published known-answer vectors
(tests/golden/philox_kat.json) and by uniformity tests.
"""
from __future__ import annotations

import math
from typing import Sequence, Tuple

M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK = 0xFFFFFFFF


def philox4x32_10(ctr: Sequence[int], key: Sequence[int]) -> Tuple[int, int, int, int]:
    c0, c1, c2, c3 = (int(x) & MASK for x in ctr)
    k0, k1 = (int(x) & MASK for x in key)
    for r in range(10):
        p0 = M0 * c0
        p1 = M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0) & MASK, p1 & MASK, ((p0 >> 32) ^ c3 ^ k1) & MASK, p0 & MASK
        if r < 9:
            k0 = (k0 + W0) & MASK
            k1 = (k1 + W1) & MASK
    return c0, c1, c2, c3


def uniform(x: int) -> float:
    return ((x >> 9) + 0.5) * 2.0 ** -23


def gumbel(x: int) -> float:
    return -math.log(-math.log(uniform(x)))
