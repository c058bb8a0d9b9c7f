"""Philox4x32-10 counter-based generator, written from its published definition.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Reference: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel Random
Numbers: As Easy as 1, 2, 3", SC'11.  Philox-4x32 keeps a 128-bit counter as
four 32-bit words and a 64-bit key as two words.  One round multiplies words 0
and 2 by two fixed odd constants, producing 64-bit products (hi, lo); the new
state is (hi1 ^ w1 ^ k0, lo1, hi0 ^ w3 ^ k1, lo0).  Between rounds the key is
advanced by a Weyl sequence (golden-ratio and sqrt(3)-1 constants).  Ten rounds.

The paper does not say how its stochastic rounding and Bernoulli masks draw
randomness; a counter-based generator makes every draw addressable by
(seed, offset, stream, element) so that the GPU and this oracle can be
compared draw for draw.  Layout used throughout:

    counter = (lo32(blk), hi32(blk), stream, 0),  blk = offset + (i >> 3)
    key     = (lo32(seed), hi32(seed))
    element i takes 16-bit half (i & 1) of output word ((i >> 1) & 3).
"""
from __future__ import annotations

import numpy as np

_MUL0 = np.uint64(0xD2511F53)
_MUL1 = np.uint64(0xCD9E8D57)
_WEYL0 = 0x9E3779B9
_WEYL1 = 0xBB67AE85
_M32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(c0, c1, c2, c3, k0: int, k1: int):
    """Ten Philox-4x32 rounds on arrays of counters; returns four uint32 arrays."""
    c0 = np.asarray(c0, dtype=np.uint64) & _M32
    c1 = np.asarray(c1, dtype=np.uint64) & _M32
    c2 = np.asarray(c2, dtype=np.uint64) & _M32
    c3 = np.asarray(c3, dtype=np.uint64) & _M32
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    key0 = int(k0) & 0xFFFFFFFF
    key1 = int(k1) & 0xFFFFFFFF
    for rnd in range(10):
        if rnd:
            key0 = (key0 + _WEYL0) & 0xFFFFFFFF
            key1 = (key1 + _WEYL1) & 0xFFFFFFFF
        p0 = c0 * _MUL0  # < 2^64: exact in uint64
        p1 = c2 * _MUL1
        hi0, lo0 = p0 >> np.uint64(32), p0 & _M32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _M32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ np.uint64(key0), lo1, hi0 ^ c3 ^ np.uint64(key1), lo0)
    return tuple(x.astype(np.uint32) for x in (c0, c1, c2, c3))


def uniforms16(seed: int, offset: int, stream: int, count: int) -> np.ndarray:
    """16-bit uniforms u_i, i = 0..count-1, of one stream (uint16 array)."""
    nblk = (int(count) + 7) // 8
    blk = np.uint64(offset) + np.arange(nblk, dtype=np.uint64)
    w = philox4x32_10(blk & _M32, blk >> np.uint64(32), np.uint64(stream), np.uint64(0),
                      int(seed) & 0xFFFFFFFF, (int(seed) >> 32) & 0xFFFFFFFF)
    words = np.stack(w, axis=-1).astype("<u4")  # [nblk][4]
    # element i = 8*blk + 2*word + half  ->  little-endian uint16 view order
    return words.view("<u2").reshape(-1)[:count].astype(np.uint16)


def philox_blocks(count: int) -> int:
    """Philox blocks one stream consumes for `count` elements."""
    return (int(count) + 7) // 8
