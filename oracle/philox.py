"""Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy
as 1, 2, 3", SC'11), in exact unsigned arithmetic on numpy uint64 arrays.

A Philox-4x32 round maps a counter (c0,c1,c2,c3) under a key (k0,k1) through
two 32x32->64 products: with (hi0,lo0) = M0*c0 and (hi1,lo1) = M1*c2 the new
counter is (hi1^c1^k0, lo1, hi0^c3^k1, lo0).  The key is advanced by the Weyl
increments between rounds; ten rounds make Philox4x32-10.  Multipliers and
increments are the published ones.

Counter and key layout used for events (one Philox call per event):
  key     = (seed & 0xffffffff, seed >> 32)
  counter = (id & 0xffffffff, id >> 32, stream, 0)
with id = counter_base + theta_index * E + k.
"""
from __future__ import annotations

import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(counter: np.ndarray, key) -> np.ndarray:
    """counter: uint32 [n, 4]; key: (k0, k1) ints.  Returns uint32 [n, 4]."""
    c = np.asarray(counter, dtype=np.uint64).reshape(-1, 4)
    c0, c1, c2, c3 = (c[:, i].copy() for i in range(4))
    k0, k1 = int(key[0]) & 0xFFFFFFFF, int(key[1]) & 0xFFFFFFFF
    for r in range(10):
        if r:
            k0 = (k0 + W0) & 0xFFFFFFFF
            k1 = (k1 + W1) & 0xFFFFFFFF
        p0 = M0 * c0            # < 2^64: exact in uint64
        p1 = M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        c0 = hi1 ^ c1 ^ np.uint64(k0)
        c1 = lo1
        c2 = hi0 ^ c3 ^ np.uint64(k1)
        c3 = lo0
    return np.stack([c0, c1, c2, c3], axis=1).astype(np.uint32)


def event_words(seed: int, ids: np.ndarray, stream: int = 0) -> np.ndarray:
    """The four Philox words of each event id (uint64 array) under `seed`."""
    ids = np.asarray(ids, dtype=np.uint64)
    ctr = np.empty((ids.size, 4), dtype=np.uint64)
    ctr[:, 0] = ids & MASK32
    ctr[:, 1] = ids >> np.uint64(32)
    ctr[:, 2] = np.uint64(stream & 0xFFFFFFFF)
    ctr[:, 3] = 0
    return philox4x32_10(ctr, (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))
