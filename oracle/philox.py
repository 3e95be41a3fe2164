"""Philox4x32-10 counter-based generator (oracle; test infrastructure only).

Published method: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw,
"Parallel random numbers: as easy as 1, 2, 3", SC'11.  Four 32-bit counter
words, two 32-bit key words, ten rounds.  Each round multiplies counter
words 0 and 2 by the constants M0, M1 to 64-bit products (hi:lo) and forms
the new counter as (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the key is
advanced by the Weyl constants W0, W1 between rounds.

Stochastic-rounding stream of this implementation (the paper asks for few-
bit-free SR, Sec. 4.3, and does not fix a generator): element i (the row-major
index of the element in the source tensor) of a tensor with identifier ``tid``
quantized with 64-bit ``seed`` uses word i & 3 of
    Philox4x32-10(counter = (j mod 2**32, j >> 32, tid, 0),
                  key = (seed mod 2**32, seed >> 32)),   j = i >> 2.
"""

import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(counter, key):
    """counter: uint32-like array [..., 4]; key: (k0, k1).  Returns the four
    output words [..., 4] as uint32."""
    c = np.asarray(counter, dtype=np.uint64) & MASK
    c0, c1, c2, c3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0 = int(key[0]) & 0xFFFFFFFF
    k1 = int(key[1]) & 0xFFFFFFFF
    for rnd in range(10):
        if rnd:
            k0 = (k0 + W0) & 0xFFFFFFFF
            k1 = (k1 + W1) & 0xFFFFFFFF
        p0 = M0 * c0            # < 2**64, exact in uint64
        p1 = M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK
        c0, c1, c2, c3 = (hi1 ^ c1 ^ np.uint64(k0), lo1,
                          hi0 ^ c3 ^ np.uint64(k1), lo0)
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def sr_words(seed, tensor_id, index):
    """The 32-bit SR word of each element index (int64 array).  Each
    distinct counter j = index >> 2 is evaluated once and its four words are
    shared by the elements 4j .. 4j+3 that use them."""
    idx = np.asarray(index, dtype=np.int64)
    uj, inv = np.unique(idx >> 2, return_inverse=True)
    j = uj.astype(np.uint64)
    ctr = np.stack([j & MASK, j >> np.uint64(32),
                    np.full_like(j, np.uint64(tensor_id & 0xFFFFFFFF)),
                    np.zeros_like(j)], axis=-1)
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    out = philox4x32_10(ctr, (seed & 0xFFFFFFFF, seed >> 32))        # [distinct j, 4]
    return out[inv.reshape(idx.shape), idx & 3]
