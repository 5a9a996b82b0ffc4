"""Philox4x64-10 counter-based generator, written from its published
definition: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel
Random Numbers: As Easy as 1, 2, 3", SC'11 (the Philox family, N=4 words of
W=64 bits, R=10 rounds).

Test infrastructure (see the package docstring).

The paper being implemented says only that the layer mask is Bernoulli per
sequence (Preliminary section, layer-dropout training equation); the generator
is a reading of it: one Philox4x64-10 block per (sample, layer, step)
counter under a (seed, 0) key, word 0 of the output used for the draw.

One round maps (c0, c1, c2, c3) under key (k0, k1) to
    (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))
and between rounds the key is bumped by the Weyl constants (W0, W1).
"""

import numpy as np

M0 = np.uint64(0xD2E7470EE14C6C93)
M1 = np.uint64(0xCA5A826395121157)
W0 = np.uint64(0x9E3779B97F4A7C15)   # golden ratio
W1 = np.uint64(0xBB67AE8584CAA73B)   # sqrt(3) - 1
ROUNDS = 10

_MASK32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def mulhilo64(a, b):
    """Full 128-bit product of two uint64 arrays, returned as (hi, lo).

    Computed from 32-bit limbs so that every partial product fits in 64 bits.
    """
    a = np.asarray(a, dtype=np.uint64)
    b = np.asarray(b, dtype=np.uint64)
    with np.errstate(over="ignore"):
        a_lo, a_hi = a & _MASK32, a >> _S32
        b_lo, b_hi = b & _MASK32, b >> _S32
        ll = a_lo * b_lo
        lh = a_lo * b_hi
        hl = a_hi * b_lo
        hh = a_hi * b_hi
        mid = (ll >> _S32) + (lh & _MASK32) + (hl & _MASK32)
        hi = hh + (lh >> _S32) + (hl >> _S32) + (mid >> _S32)
        lo = (mid << _S32) | (ll & _MASK32)
    return hi, lo


def philox4x64_10(c0, c1, c2, c3, k0, k1):
    """Return the four output words of Philox4x64-10 for the given counter
    words (c0 least significant) and key words.  Arguments broadcast."""
    c0, c1, c2, c3, k0, k1 = np.broadcast_arrays(
        *[np.asarray(v, dtype=np.uint64) for v in (c0, c1, c2, c3, k0, k1)])
    c0, c1, c2, c3 = c0.copy(), c1.copy(), c2.copy(), c3.copy()
    k0, k1 = k0.copy(), k1.copy()
    with np.errstate(over="ignore"):
        for rnd in range(ROUNDS):
            if rnd > 0:
                k0 = k0 + W0
                k1 = k1 + W1
            hi0, lo0 = mulhilo64(M0, c0)
            hi1, lo1 = mulhilo64(M1, c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def block_words(sample, layer, step, seed, c3=0):
    """All four output words for counter (sample, layer, step, c3) and key
    (seed, 0).  Sub-layer masks use words 0 and 1 of one block; per-batch
    draws use c3 = 1 (so they never share a block with a per-sequence draw)."""
    return philox4x64_10(sample, layer, step, c3, seed, 0)


def mask_word(sample, layer, step, seed):
    """The 64-bit draw for one (sample, layer, step) under `seed`: word 0 of
    Philox4x64-10 with counter (sample, layer, step, 0) and key (seed, 0)."""
    w0, _, _, _ = philox4x64_10(sample, layer, step, 0, seed, 0)
    return w0
