"""Exact-k uniform draw without replacement (oracle; test infrastructure only).

The paper samples each seed's neighbours uniformly from the (causal) pool
(Methods, "Sampling Modes: Stochastic and Structural", Stochastic item) with
``torch.randint`` and asks for a given density.  Reading taken here: the draw
is *exact-count* -- ``k`` distinct keys, uniform over all k-subsets of the
pool -- so that the density is met exactly per row and no per-seed dedupe is
needed.  It is realised by a keyed pseudo-random permutation ``P`` of
``[0, n)`` and taking ``{P(0), ..., P(k-1)}``.

``P`` is a balanced Feistel network on ``m``-bit words,
``m = max(2, bitlen(n-1))`` rounded up to even, half width ``h = m/2``, six
rounds.  Round ``r`` maps ``(L, R) -> (R, L xor (F(R xor rk_r) & (2^h-1)))``
with ``F`` the MurmurHash3 32-bit finaliser ``fmix32`` (Appleby, public
domain).  Values ``>= n`` are cycle-walked (re-encrypted until they fall in
range), which restricts a permutation of ``[0, 2^m)`` to one of ``[0, n)``
(Black and Rogaway, "Ciphers with arbitrary finite domains", 2002).

Pinned by: ``fmix32`` against scikit-learn's MurmurHash3 of the empty string
(which reduces to ``fmix32(seed)``); exhaustive bijectivity; distinctness and
range of cycle-walked draws; chi-square uniformity of inclusion over keys.
The particular permutation is a definitional choice (any uniform draw realises
the paper's sampling); the GPU reproduces it bit for bit.
"""

import numpy as np

_M32 = np.uint64(0xFFFFFFFF)
FMIX_C1 = np.uint64(0x85EBCA6B)
FMIX_C2 = np.uint64(0xC2B2AE35)
ROUNDS = 6


def fmix32(h):
    """MurmurHash3 32-bit finaliser on uint64 arrays holding 32-bit values."""
    h = np.asarray(h, dtype=np.uint64) & _M32
    h = h ^ (h >> np.uint64(16))
    h = (h * FMIX_C1) & _M32
    h = h ^ (h >> np.uint64(13))
    h = (h * FMIX_C2) & _M32
    h = h ^ (h >> np.uint64(16))
    return h


def domain_bits(n):
    """Feistel word width m for pool sizes n (even, at least 2).

    Works elementwise on integer arrays; n = 1 gives 2 (unused: P is 0 there).
    """
    n = np.asarray(n, dtype=np.int64)
    m = np.zeros(n.shape, dtype=np.int64)
    v = np.maximum(n - 1, 0)
    while (v > 0).any():          # bit length of n - 1
        m += (v > 0)
        v >>= 1
    m = np.maximum(m, 2)
    return m + (m & 1)


def feistel(x, rk, m):
    """One application of the six-round Feistel permutation of [0, 2^m).

    x: uint64 array of values < 2^m.  rk: uint64 array (..., 6) of round keys
    with leading shape equal to x's.  m: even word widths, broadcast with x.
    """
    x = np.asarray(x, dtype=np.uint64)
    h = np.broadcast_to(np.asarray(m, dtype=np.uint64) // np.uint64(2), x.shape)
    mask = (np.uint64(1) << h) - np.uint64(1)
    left = x >> h
    right = x & mask
    for r in range(ROUNDS):
        f = fmix32(right ^ rk[..., r]) & mask
        left, right = right, left ^ f
    return (left << h) | right


def permute(j, rk, n):
    """P(j) for the keyed permutation of [0, n), by cycle walking.

    j: uint64 array of values < n.  rk: round keys (j.shape + (6,)) or one key
    set (6,).  n: pool sizes >= 1, broadcast with j.
    """
    j = np.asarray(j, dtype=np.uint64)
    n = np.broadcast_to(np.asarray(n, dtype=np.uint64), j.shape)
    rk = np.broadcast_to(np.asarray(rk, dtype=np.uint64), j.shape + (ROUNDS,))
    m = domain_bits(n.astype(np.int64))
    x = feistel(j, rk, m)
    bad = x >= n
    while bad.any():
        x[bad] = feistel(x[bad], rk[bad], m[bad])
        bad = x >= n
    return np.where(n == np.uint64(1), np.uint64(0), x)


def draw(k, n, rk):
    """The k keys {P(0), ..., P(k-1)} drawn from [0, n) (distinct, unsorted)."""
    if k <= 0 or n <= 0:
        return np.zeros(0, dtype=np.uint64)
    return permute(np.arange(k, dtype=np.uint64), np.asarray(rk, dtype=np.uint64), n)
