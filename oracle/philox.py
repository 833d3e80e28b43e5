"""Philox counter-based block functions, written from their published definition.

Source: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC'11 -- the Philox-4xW-R family.  One round maps
the counter (c0, c1, c2, c3) under key (k0, k1) to

    (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))

where hi/lo are the upper/lower W bits of the 2W-bit product, and the key is
bumped by the Weyl constants (C0, C1) between rounds.  R = 10 rounds.

The dropout masks of the method (§3.3 Model Pack: "m dropout masks with m
different rates") need a random source that the GPU path can reproduce bit for
bit, so the masks are defined on Philox4x32-10 (the GPU's 32-bit integer
multiplier makes the 32-bit variant the cheaper one); the 64-bit variant is
implemented with the same round structure only so that it can be pinned
against numpy's independent ``np.random.Philox`` (which is Philox4x64-10).
"""
import numpy as np

PHILOX4x32 = dict(W=32, M=(0xD2511F53, 0xCD9E8D57), C=(0x9E3779B9, 0xBB67AE85))
PHILOX4x64 = dict(W=64, M=(0xD2E7470EE14C6C93, 0xCA5A826395121157),
                  C=(0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B))


def philox_scalar(ctr, key, W, M, C, rounds=10):
    """Philox-4xW on Python integers (any W); returns the 4 output words."""
    mask = (1 << W) - 1
    c0, c1, c2, c3 = (int(x) & mask for x in ctr)
    k0, k1 = (int(x) & mask for x in key)
    for _ in range(rounds):
        p0 = M[0] * c0
        p1 = M[1] * c2
        c0, c1, c2, c3 = ((p1 >> W) ^ c1 ^ k0, p1 & mask,
                          (p0 >> W) ^ c3 ^ k1, p0 & mask)
        k0 = (k0 + C[0]) & mask
        k1 = (k1 + C[1]) & mask
    return [c0, c1, c2, c3]


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10.

    Counter words c0..c3 are broadcastable integer arrays (< 2**32), the key
    words k0, k1 are Python ints.  Returns four uint32 arrays.  The 32x32->64
    bit products are formed exactly in uint64.
    """
    m = np.uint64(0xFFFFFFFF)
    c0, c1, c2, c3 = np.broadcast_arrays(*(np.asarray(c, dtype=np.uint64) for c in (c0, c1, c2, c3)))
    c0, c1, c2, c3 = (x.copy() for x in (c0, c1, c2, c3))
    M0, M1 = (np.uint64(v) for v in PHILOX4x32["M"])
    C0, C1 = PHILOX4x32["C"]
    k0 = int(k0) & 0xFFFFFFFF
    k1 = int(k1) & 0xFFFFFFFF
    for _ in range(10):
        p0 = M0 * c0
        p1 = M1 * c2
        n0 = (p1 >> np.uint64(32)) ^ c1 ^ np.uint64(k0)
        n1 = p1 & m
        n2 = (p0 >> np.uint64(32)) ^ c3 ^ np.uint64(k1)
        n3 = p0 & m
        c0, c1, c2, c3 = n0, n1, n2, n3
        k0 = (k0 + C0) & 0xFFFFFFFF
        k1 = (k1 + C1) & 0xFFFFFFFF
    return tuple(x.astype(np.uint32) for x in (c0, c1, c2, c3))
