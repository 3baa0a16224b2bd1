"""Philox4x32-10 counter-based generator (oracle side).

Written from the description in Salmon, Moraes, Dror and Shaw, "Parallel
Random Numbers: As Easy as 1, 2, 3" (SC'11), Section 5: a 4x32-bit counter and
a 2x32-bit key; each of the 10 rounds multiplies counter words 0 and 2 by two
fixed 32-bit multipliers, takes the high and low halves of the 64-bit products
and permutes/XORs them with the other two words and the round key; the key is
bumped by two Weyl constants between rounds.

The refusal-gated decoding method draws one uniform per sampled token; here
that uniform is the top 24 bits of word 0 scaled by 2^-24, so it is exactly
representable in fp32 and fp64 alike.

Pinned by: published known-answer vectors of the SC'11 authors' Random123
distribution (tests/golden/philox4x32_10_kat.txt), an independent host
compile of rocRAND's philox4x32_10 engine, and a uniformity chi-square test.
"""
from __future__ import annotations

import numpy as np

MULT = (0xD2511F53, 0xCD9E8D57)   # round multipliers for words 0 and 2
WEYL = (0x9E3779B9, 0xBB67AE85)   # key increments (golden ratio, sqrt(3)-1)
_M32 = 0xFFFFFFFF


def philox4x32_10_int(counter, key):
    """Scalar Philox4x32-10 on Python ints.  counter: 4 words, key: 2 words."""
    c0, c1, c2, c3 = (int(x) & _M32 for x in counter)
    k0, k1 = (int(x) & _M32 for x in key)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + WEYL[0]) & _M32
            k1 = (k1 + WEYL[1]) & _M32
        p0 = MULT[0] * c0
        p1 = MULT[1] * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0, p1 & _M32,
                          (p0 >> 32) ^ c3 ^ k1, p0 & _M32)
    return c0, c1, c2, c3


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10 on numpy arrays (broadcasting); returns 4 uint64
    arrays holding 32-bit words."""
    m = np.uint64(_M32)
    c0, c1, c2, c3, k0, k1 = (np.asarray(x, dtype=np.uint64) & m
                              for x in (c0, c1, c2, c3, k0, k1))
    c0, c1, c2, c3, k0, k1 = np.broadcast_arrays(c0, c1, c2, c3, k0, k1)
    s32 = np.uint64(32)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + np.uint64(WEYL[0])) & m
            k1 = (k1 + np.uint64(WEYL[1])) & m
        p0 = np.uint64(MULT[0]) * c0          # < 2^64: exact in uint64
        p1 = np.uint64(MULT[1]) * c2
        c0, c1, c2, c3 = ((p1 >> s32) ^ c1 ^ k0, p1 & m, (p0 >> s32) ^ c3 ^ k1, p0 & m)
    return c0, c1, c2, c3


def split_seed(seed):
    """64-bit seed -> (key word 0, key word 1) = (low 32 bits, high 32 bits)."""
    s = np.asarray(seed, dtype=np.uint64)
    return s & np.uint64(_M32), s >> np.uint64(32)


def uniform(seed, ctr, stream=0):
    """The draw used by the sampler: key = seed (lo, hi), counter =
    (ctr, stream, 0, 0); u = (word0 >> 8) * 2^-24 in [0, 1), as float64."""
    k0, k1 = split_seed(seed)
    x0, _, _, _ = philox4x32_10(ctr, stream, 0, 0, k0, k1)
    return (x0 >> np.uint64(8)).astype(np.float64) * 2.0 ** -24
