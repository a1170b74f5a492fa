"""Philox4x32-10 counter-based generator, written from its published definition.

TEST INFRASTRUCTURE ONLY.  This module belongs to the CPU oracle; only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it.  The
GPU library carries its own, independent implementation.

Reference: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC'11 -- the Philox-4x32 bijection with ten
rounds.  One round takes a 4-word counter (c0, c1, c2, c3) and a 2-word key
(k0, k1); it forms the 64-bit products M0*c0 and M1*c2 and outputs

    (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))

and between rounds the key is advanced by the Weyl constants (W0, W1).

The NaCl paper asks for random eviction with a different seed for every
attention head and layer (Section 1 and Section 6.3, head-wise eviction).  The
counter-based generator makes that draw a pure function of
(seed; token block, head, batch row, layer), independent of how the work is
split across threads.

Parity status: pinned against an independent implementation (rocRAND's
host-callable Philox4x32-10) by the CPU test suite, plus statistical checks.
"""

import numpy as np

PHILOX_M0 = np.uint64(0xD2511F53)
PHILOX_M1 = np.uint64(0xCD9E8D57)
PHILOX_W0 = np.uint32(0x9E3779B9)
PHILOX_W1 = np.uint32(0xBB67AE85)
_LO32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def philox4x32_10(c0, c1, c2, c3, k0, k1, rounds=10):
    """Apply the Philox4x32 bijection (default ten rounds) element-wise.

    All arguments are broadcastable unsigned 32-bit arrays (or Python ints);
    returns a tuple of four uint32 arrays, the output words in order.
    """
    c0 = np.asarray(c0, dtype=np.uint32)
    c1 = np.asarray(c1, dtype=np.uint32)
    c2 = np.asarray(c2, dtype=np.uint32)
    c3 = np.asarray(c3, dtype=np.uint32)
    k0 = np.asarray(k0, dtype=np.uint32)
    k1 = np.asarray(k1, dtype=np.uint32)
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    with np.errstate(over="ignore"):
        for r in range(rounds):
            if r:
                k0 = (k0 + PHILOX_W0).astype(np.uint32)
                k1 = (k1 + PHILOX_W1).astype(np.uint32)
            p0 = PHILOX_M0 * c0.astype(np.uint64)
            p1 = PHILOX_M1 * c2.astype(np.uint64)
            hi0 = (p0 >> _S32).astype(np.uint32)
            lo0 = (p0 & _LO32).astype(np.uint32)
            hi1 = (p1 >> _S32).astype(np.uint32)
            lo1 = (p1 & _LO32).astype(np.uint32)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def seed_to_key(seed):
    """Split a 64-bit seed into the Philox key words (low word first)."""
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return np.uint32(seed & 0xFFFFFFFF), np.uint32(seed >> 32)


def token_words(seed, layer, b, h, L):
    """The 32-bit random word owned by each token j in [0, L) of one head.

    Counter convention: (floor(j/4), h, b, layer), key = seed; token j takes
    output word j mod 4.  Returns a uint32 array of length L.
    """
    nq = (L + 3) // 4
    q = np.arange(nq, dtype=np.uint64).astype(np.uint32)
    k0, k1 = seed_to_key(seed)
    w = philox4x32_10(q, np.uint32(h), np.uint32(b), np.uint32(layer), k0, k1)
    out = np.stack(w, axis=1).reshape(-1)
    return out[:L]


def open_unit(words):
    """Map 32-bit words to doubles strictly inside (0, 1): (x + 1/2) / 2^32.

    Both operations are exact in binary64, so every implementation that follows
    this definition produces identical doubles.
    """
    return (np.asarray(words, dtype=np.float64) + 0.5) * (2.0 ** -32)
