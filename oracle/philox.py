"""Philox4x32-10, written from its published definition (oracle; test-only).

Source of the definition: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw,
"Parallel Random Numbers: As Easy as 1, 2, 3", SC'11.  The paper this library
implements says only that each perturbation is regenerated from an integer
seed (Section 3; Appendix D.6); the generator itself is this published one.

One call maps a 128-bit counter (c0, c1, c2, c3) and a 64-bit key (k0, k1),
all as 32-bit words, to four 32-bit output words.  A round is

    (hi0, lo0) = 64-bit product of 0xD2511F53 and c0
    (hi1, lo1) = 64-bit product of 0xCD9E8D57 and c2
    (c0, c1, c2, c3) <- (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0)

and between consecutive rounds the key is bumped by the Weyl constants
k0 += 0x9E3779B9, k1 += 0xBB67AE85 (mod 2^32).  Ten rounds make one call.

Pins (tests/test_oracle_philox.py): word-for-word agreement with two
independent source-available implementations of the same generator (PyTorch's
host philox engine and rocRAND's), compiled as tiny host harnesses, on random
keys and counters; and agreement of the vectorised and big-integer versions.
"""

import numpy as np

MASK32 = 0xFFFFFFFF
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
PHILOX_ROUNDS = 10


def philox4x32_10(ctr, key):
    """Vectorised Philox4x32-10.

    ctr: sequence of four integer arrays (or scalars), the counter words
         c0..c3, each holding values in [0, 2^32).
    key: sequence of two integers or integer arrays, the key words k0, k1.
    Returns a (4, n) uint64 array holding the four 32-bit output words.

    Products of two 32-bit values fit in 64 bits, so uint64 arithmetic is exact.
    """
    c = [np.atleast_1d(np.asarray(w, dtype=np.uint64)) & np.uint64(MASK32)
         for w in ctr]
    n = max(x.shape[0] for x in c)
    c = [np.broadcast_to(x, (n,)).copy() for x in c]
    k0 = np.broadcast_to(np.asarray(key[0], dtype=np.uint64), (n,)) & np.uint64(MASK32)
    k1 = np.broadcast_to(np.asarray(key[1], dtype=np.uint64), (n,)) & np.uint64(MASK32)
    m0 = np.uint64(PHILOX_M0)
    m1 = np.uint64(PHILOX_M1)
    mask = np.uint64(MASK32)
    sh = np.uint64(32)
    c0, c1, c2, c3 = c
    for r in range(PHILOX_ROUNDS):
        if r > 0:
            k0 = (k0 + np.uint64(PHILOX_W0)) & mask
            k1 = (k1 + np.uint64(PHILOX_W1)) & mask
        p0 = m0 * c0
        p1 = m1 * c2
        hi0, lo0 = p0 >> sh, p0 & mask
        hi1, lo1 = p1 >> sh, p1 & mask
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3])


def philox4x32_10_bigint(ctr, key):
    """The same generator for one counter, with Python integers throughout.

    A second, deliberately naive rendering used to cross-check the vectorised
    one on small inputs.  Returns a tuple of four ints.
    """
    c0, c1, c2, c3 = (int(x) & MASK32 for x in ctr)
    k0, k1 = int(key[0]) & MASK32, int(key[1]) & MASK32
    for r in range(PHILOX_ROUNDS):
        if r:
            k0 = (k0 + PHILOX_W0) % (1 << 32)
            k1 = (k1 + PHILOX_W1) % (1 << 32)
        prod0 = PHILOX_M0 * c0
        prod1 = PHILOX_M1 * c2
        hi0, lo0 = divmod(prod0, 1 << 32)
        hi1, lo1 = divmod(prod1, 1 << 32)
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return (c0, c1, c2, c3)
