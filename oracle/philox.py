"""Philox4x32-10 (Salmon, Moraes, Dror, Shaw: "Parallel Random Numbers: As Easy
as 1, 2, 3", SC'11, Sec. 3 and Table 2).

The sampler's random c-subsets (Alg. 3, "rand(c)") need a generator that every
row can evaluate independently; a counter-based generator gives exactly that.

One round maps counter (c0, c1, c2, c3) and key (k0, k1) to
    (hi(B*c2) ^ c1 ^ k0,  lo(B*c2),  hi(A*c0) ^ c3 ^ k1,  lo(A*c0))
with A = 0xD2511F53, B = 0xCD9E8D57 and hi/lo the halves of the 64-bit product.
The key is bumped by the Weyl constants (0x9E3779B9, 0xBB67AE85) between
rounds; ten rounds in total.

Pinned by the published known-answer vectors (tests/golden/philox4x32_10_kat.txt).
"""
import numpy as np

MUL_A = 0xD2511F53
MUL_B = 0xCD9E8D57
WEYL_0 = 0x9E3779B9
WEYL_1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32_10(ctr, key):
    """Scalar Philox4x32-10.  ctr: 4 ints, key: 2 ints -> list of 4 ints."""
    c0, c1, c2, c3 = (int(x) & MASK32 for x in ctr)
    k0, k1 = (int(x) & MASK32 for x in key)
    for _ in range(10):
        pa = MUL_A * c0
        pb = MUL_B * c2
        c0, c1, c2, c3 = ((pb >> 32) ^ c1 ^ k0, pb & MASK32,
                          (pa >> 32) ^ c3 ^ k1, pa & MASK32)
        k0 = (k0 + WEYL_0) & MASK32
        k1 = (k1 + WEYL_1) & MASK32
    return [c0, c1, c2, c3]


def philox4x32_10_np(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10 over numpy arrays (broadcasting), same rounds.

    Arguments are integer arrays or scalars holding 32-bit values; the result
    is a tuple of four uint64 arrays holding 32-bit values.
    """
    u = np.uint64
    c0, c1, c2, c3 = (np.asarray(x, dtype=np.uint64) & u(MASK32) for x in (c0, c1, c2, c3))
    k0 = np.asarray(k0, dtype=np.uint64) & u(MASK32)
    k1 = np.asarray(k1, dtype=np.uint64) & u(MASK32)
    c0, c1, c2, c3, k0, k1 = np.broadcast_arrays(c0, c1, c2, c3, k0, k1)
    c0, c1, c2, c3, k0, k1 = (x.copy() for x in (c0, c1, c2, c3, k0, k1))
    for _ in range(10):
        pa = u(MUL_A) * c0          # < 2^64, exact in uint64
        pb = u(MUL_B) * c2
        n0 = (pb >> u(32)) ^ c1 ^ k0
        n1 = pb & u(MASK32)
        n2 = (pa >> u(32)) ^ c3 ^ k1
        n3 = pa & u(MASK32)
        c0, c1, c2, c3 = n0, n1, n2, n3
        k0 = (k0 + u(WEYL_0)) & u(MASK32)
        k1 = (k1 + u(WEYL_1)) & u(MASK32)
    return c0, c1, c2, c3
