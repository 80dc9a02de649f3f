"""Philox4x64-10 counter-based generator, written from its published definition.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import this module;
only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` use it.

Definition followed: Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As
Easy as 1, 2, 3" (SC'11), Philox-4x64 with R = 10 rounds.  One round maps the
counter (c0, c1, c2, c3) under key (k0, k1) to

    (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))

where hi/lo are the two halves of the 128-bit product; the key is advanced by
the Weyl constants (W0, W1) between rounds.  The multipliers and Weyl
constants are the ones that paper publishes for the 4x64 variant.

The paper under study (Partial FC) only asks for "sampling without
replacement" and names no generator; using a counter-based generator keyed by
the global class id is this implementation's reading (one key per class, no
state, independent of how classes are sharded).

Pinned in tests by the known-answer vectors distributed with the SC'11 paper's
reference library (tests/golden/philox4x64_10_kat.txt) and by an independent
library implementation (numpy.random.Philox).
"""

import numpy as np

M0 = 0xD2E7470EE14C6C93
M1 = 0xCA5A826395121157
W0 = 0x9E3779B97F4A7C15
W1 = 0xBB67AE8584CAA73B
ROUNDS = 10
_MASK64 = (1 << 64) - 1


def philox4x64_scalar(ctr, key, rounds=ROUNDS):
    """One Philox4x64 block with Python integers (exact 128-bit products)."""
    c0, c1, c2, c3 = (int(v) & _MASK64 for v in ctr)
    k0, k1 = (int(v) & _MASK64 for v in key)
    for r in range(rounds):
        if r > 0:
            k0 = (k0 + W0) & _MASK64
            k1 = (k1 + W1) & _MASK64
        p0 = M0 * c0
        p1 = M1 * c2
        hi0, lo0 = p0 >> 64, p0 & _MASK64
        hi1, lo1 = p1 >> 64, p1 & _MASK64
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return (c0, c1, c2, c3)


def _mulhilo64(a, b):
    """Vectorised 64x64 -> (hi, lo) product using 32-bit limbs in uint64."""
    a = a.astype(np.uint64)
    b = np.uint64(b)
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a_lo, a_hi = a & m32, a >> s32
    b_lo, b_hi = b & m32, b >> s32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> s32) + (lh & m32) + (hl & m32)
    lo = (ll & m32) | ((mid & m32) << s32)
    hi = hh + (lh >> s32) + (hl >> s32) + (mid >> s32)
    return hi, lo


def philox4x64_blocks(c0, key, rounds=ROUNDS):
    """Philox4x64 of counters (c0[i], 0, 0, 0) under one key, vectorised.

    Returns a uint64 array of shape (len(c0), 4): word w of block i.
    """
    with np.errstate(over="ignore"):
        x0 = np.asarray(c0, dtype=np.uint64).copy()
        x1 = np.zeros_like(x0)
        x2 = np.zeros_like(x0)
        x3 = np.zeros_like(x0)
        k0 = np.uint64(int(key[0]) & _MASK64)
        k1 = np.uint64(int(key[1]) & _MASK64)
        for r in range(rounds):
            if r > 0:
                k0 = np.uint64((int(k0) + W0) & _MASK64)
                k1 = np.uint64((int(k1) + W1) & _MASK64)
            hi0, lo0 = _mulhilo64(x0, M0)
            hi1, lo1 = _mulhilo64(x2, M1)
            x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
        return np.stack([x0, x1, x2, x3], axis=1)


def class_keys(seed, global_ids):
    """Random 64-bit key of each global class id g.

    Reading of the paper's unspecified sampler: key(g) is word (g mod 4) of
    the Philox4x64-10 block with counter (floor(g/4), 0, 0, 0) and key
    (seed, 0).  Keys depend only on (seed, g), so every shard draws the same
    key for a class whatever its offset.
    """
    g = np.asarray(global_ids, dtype=np.int64)
    if g.size == 0:
        return np.zeros(0, dtype=np.uint64)
    blk = g // 4
    first = int(blk.min())
    words = philox4x64_blocks(np.arange(first, int(blk.max()) + 1), (seed, 0))
    return words[blk - first, g % 4].astype(np.uint64)
