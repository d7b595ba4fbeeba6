"""Philox4x64-10 counter-based generator (oracle; test infrastructure only).

Follows the published definition of Salmon, Moraes, Dror and Shaw, "Parallel
random numbers: as easy as 1, 2, 3" (SC'11): a 4-word, 64-bit-lane counter is
pushed through ten rounds of two 64x64->128 multiplies, with a Weyl-sequence key
schedule between rounds.

The paper draws each seed's indices with ``torch.randint`` (Methods,
"Memory-Bounded Geometry Generation").  Any uniform generator realises that
draw; a counter-based one lets every (seed, layer, kv-head, query) row be drawn
independently, in any order, on either side of the parity check.

Reading taken here: the row key is derived from Philox with
``key = (seed, 0)`` and ``counter = (query, kv_head, layer, 0)``; the four
64-bit outputs are split into eight 32-bit words, low half first, which feed
the Feistel round keys (see ``prp``).

Pinned by: known-answer equality with ``numpy.random.Philox`` (an independent
library implementation of the same published algorithm).
"""

import numpy as np

# Published Philox4x64 multipliers and Weyl key increments.
M0 = np.uint64(0xD2E7470EE14C6C93)
M1 = np.uint64(0xCA5A826395121157)
W0 = np.uint64(0x9E3779B97F4A7C15)
W1 = np.uint64(0xBB67AE8584CAA73B)
_LO32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def mulhilo64(a, b):
    """Full 128-bit product of uint64 arrays, returned as (hi, lo) uint64.

    Schoolbook product over 32-bit halves; no partial sum overflows 64 bits.
    """
    a = np.asarray(a, dtype=np.uint64)
    b = np.asarray(b, dtype=np.uint64)
    a0, a1 = a & _LO32, a >> _S32
    b0, b1 = b & _LO32, b >> _S32
    with np.errstate(over="ignore"):
        p00 = a0 * b0
        p10 = a1 * b0
        p01 = a0 * b1
        p11 = a1 * b1
        mid = (p00 >> _S32) + (p10 & _LO32) + p01
        hi = p11 + (p10 >> _S32) + (mid >> _S32)
        lo = a * b
    return hi, lo


def philox4x64_10(counter, key):
    """Philox4x64-10 block function.

    counter: sequence of four uint64 arrays (broadcastable), key: two uint64
    arrays.  Returns four uint64 arrays.
    """
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) for c in counter)
    k0, k1 = (np.asarray(k, dtype=np.uint64) for k in key)
    c0, c1, c2, c3, k0, k1 = np.broadcast_arrays(c0, c1, c2, c3, k0, k1)
    c0, c1, c2, c3 = c0.copy(), c1.copy(), c2.copy(), c3.copy()
    k0, k1 = k0.copy(), k1.copy()
    for rnd in range(10):
        if rnd > 0:
            with np.errstate(over="ignore"):
                k0 = k0 + W0
                k1 = k1 + W1
        hi0, lo0 = mulhilo64(M0, c0)
        hi1, lo1 = mulhilo64(M1, c2)
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def row_round_keys(seed, q, kv_head, layer):
    """The eight 32-bit words of one (seed, layer, kv_head, query) row.

    All arguments broadcast.  Returns a uint64 array of shape (..., 8) whose
    values are < 2**32.
    """
    seed = np.asarray(seed, dtype=np.uint64)
    o = philox4x64_10(
        (np.asarray(q, dtype=np.uint64), np.asarray(kv_head, dtype=np.uint64),
         np.asarray(layer, dtype=np.uint64), np.uint64(0)),
        (seed, np.uint64(0)),
    )
    words = []
    for w in o:
        words.append(w & _LO32)
        words.append(w >> _S32)
    return np.stack(words, axis=-1)
