"""Philox4x32-10 counter-based generator (test infrastructure only).

Definition: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC'11, section 4.2 (Philox): a 4-word
counter and a 2-word key; each round multiplies words 0 and 2 by fixed odd
constants, swaps the high/low halves into a new word order xored with the key,
and bumps the key by the Weyl increments.  Ten rounds.

The paper being reproduced (arXiv 2609.04010) does not say how its noise is
drawn; the counter layout below is the reading adopted here (see `counter`).

Pinned by the Random123 known-answer vectors (tests/golden/philox_kat.txt) and
by agreement of the two implementations here (scalar Python ints vs numpy).
"""
import numpy as np

_M0 = 0xD2511F53
_M1 = 0xCD9E8D57
_W0 = 0x9E3779B9
_W1 = 0xBB67AE85
_MASK = 0xFFFFFFFF

# Counter word 3 selects an independent stream per use of randomness.
STREAM_TOP = 0      # group-level Gumbels of the two-level sampler
STREAM_CLASS = 1    # per-class Gumbels of the two-level sampler
STREAM_LATENT = 2   # Gaussian latents (uniform-state start / probes)
STREAM_PARAM = 3    # parameter initialisation
STREAM_VERIFY = 4   # acceptance uniforms of speculative verification
STREAM_GROUP_U = 5  # per-group uniforms of the inverse-CDF level 2 of the two-level sampler


def philox_scalar(ctr, key, rounds=10):
    """One Philox4x32 block with plain Python integers; returns 4 words."""
    c0, c1, c2, c3 = (int(v) & _MASK for v in ctr)
    k0, k1 = (int(v) & _MASK for v in key)
    for _ in range(rounds):
        p0 = _M0 * c0
        p1 = _M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0) & _MASK, p1 & _MASK, \
                         ((p0 >> 32) ^ c3 ^ k1) & _MASK, p0 & _MASK
        k0 = (k0 + _W0) & _MASK
        k1 = (k1 + _W1) & _MASK
    return c0, c1, c2, c3


def philox(c0, c1, c2, c3, k0, k1, rounds=10):
    """Vectorised Philox4x32 over broadcastable uint32-valued arrays.

    Products are formed in uint64 (a 32x32-bit product fits exactly).
    Returns four uint32 arrays.
    """
    u64 = np.uint64
    c0, c1, c2, c3, k0, k1 = np.broadcast_arrays(
        *(np.asarray(v, dtype=np.uint64) & u64(_MASK) for v in (c0, c1, c2, c3, k0, k1)))
    c0, c1, c2, c3 = c0.copy(), c1.copy(), c2.copy(), c3.copy()
    k0, k1 = k0.copy(), k1.copy()
    m0, m1, mask, s32 = u64(_M0), u64(_M1), u64(_MASK), u64(32)
    for _ in range(rounds):
        p0 = m0 * c0
        p1 = m1 * c2
        n0 = ((p1 >> s32) ^ c1 ^ k0) & mask
        n1 = p1 & mask
        n2 = ((p0 >> s32) ^ c3 ^ k1) & mask
        n3 = p0 & mask
        c0, c1, c2, c3 = n0, n1, n2, n3
        k0 = (k0 + u64(_W0)) & mask
        k1 = (k1 + u64(_W1)) & mask
    return tuple(v.astype(np.uint32) for v in (c0, c1, c2, c3))


def key_of(seed):
    """Split a 64-bit seed into the two key words (low word first)."""
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return seed & _MASK, seed >> 32


def counter_words(seed, stream, step, row, index):
    """The uint32 word assigned to (stream, step, row, index).

    Counter = (index >> 2, row, step, stream); the block's word (index & 3) is
    returned.  `row`, `index` broadcast; `step` and `stream` are scalars.
    """
    k0, k1 = key_of(seed)
    row = np.asarray(row, dtype=np.uint64)
    index = np.asarray(index, dtype=np.uint64)
    row, index = np.broadcast_arrays(row, index)
    w = philox(index >> np.uint64(2), row, np.uint64(step), np.uint64(stream), k0, k1)
    sel = (index & np.uint64(3)).astype(np.int64)
    out = np.choose(sel, w)
    return out.astype(np.uint32)
