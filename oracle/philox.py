"""Philox4x32-10 counter-based generator, written from its published definition.

TEST INFRASTRUCTURE. Part of the CPU oracle: only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import it. It shares no code
with the HIP library.

Published method: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw,
"Parallel random numbers: as easy as 1, 2, 3", SC'11 (Philox family,
section 5).  Philox4x32 acts on a 128-bit counter (four 32-bit words
c0..c3) under a 64-bit key (k0, k1).  One round multiplies c0 and c2 by the
two round multipliers, splits each 64-bit product into high and low halves,
and rearranges the words so that

    c0' = hi(M1*c2) ^ c1 ^ k0      c1' = lo(M1*c2)
    c2' = hi(M0*c0) ^ c3 ^ k1      c3' = lo(M0*c0)

Between rounds the key is advanced by the Weyl constants (golden ratio and
sqrt(3)-1 in 32-bit fixed point).  Ten rounds give Philox4x32-10.

The paper does not specify a generator; its randomized sign operators
(Section 3.1, Eqs. (9) and (10)) only need independent uniforms.  How the
stream is keyed per element is fixed in ``dsm_oracle.randomized_sign_uniforms``.
"""
import numpy as np

M0 = 0xD2511F53
M1 = 0xCD9E8D57
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32_10_scalar(ctr, key):
    """One block of Philox4x32-10 with plain Python integers.

    ctr: four 32-bit words (c0, c1, c2, c3); key: two 32-bit words (k0, k1).
    Returns the four 32-bit output words.  Slow; used for small cases and as
    the cross-check of the vectorised version.
    """
    c0, c1, c2, c3 = (int(v) & MASK32 for v in ctr)
    k0, k1 = (int(v) & MASK32 for v in key)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + W0) & MASK32
            k1 = (k1 + W1) & MASK32
        p0 = M0 * c0
        p1 = M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0, p1 & MASK32,
                          (p0 >> 32) ^ c3 ^ k1, p0 & MASK32)
    return (c0, c1, c2, c3)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10 over numpy arrays of counters.

    c0..c3: integer arrays (or scalars) broadcast together, each word < 2**32.
    k0, k1: Python ints < 2**32 (the key is the same for every block).
    Returns four uint32 arrays.  64-bit products of two 32-bit words fit in
    uint64 exactly, so the high/low split is exact.
    """
    c0, c1, c2, c3 = np.broadcast_arrays(*(np.asarray(v, dtype=np.uint64)
                                           for v in (c0, c1, c2, c3)))
    c0, c1, c2, c3 = (v.copy() for v in (c0, c1, c2, c3))
    m32 = np.uint64(MASK32)
    sh = np.uint64(32)
    k0 = int(k0) & MASK32
    k1 = int(k1) & MASK32
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + W0) & MASK32
            k1 = (k1 + W1) & MASK32
        p0 = np.uint64(M0) * c0
        p1 = np.uint64(M1) * c2
        n0 = (p1 >> sh) ^ c1 ^ np.uint64(k0)
        n1 = p1 & m32
        n2 = (p0 >> sh) ^ c3 ^ np.uint64(k1)
        n3 = p0 & m32
        c0, c1, c2, c3 = n0, n1, n2, n3
    return tuple(v.astype(np.uint32) for v in (c0, c1, c2, c3))
