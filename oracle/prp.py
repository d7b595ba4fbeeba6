"""Exact-k uniform draw without replacement (oracle; test infrastructure only).

The paper samples each seed's neighbours uniformly from the (causal) pool
(Methods, "Sampling Modes: Stochastic and Structural", Stochastic item) with
``torch.randint`` and asks for a given density.  Reading taken here: the draw
is *exact-count* -- ``k`` distinct keys, uniform over all k-subsets of the
pool -- so that the density is met exactly per row and no per-seed dedupe is
needed.  It is realised by a keyed pseudo-random permutation ``P`` of
``[0, n)`` and taking ``{P(0), ..., P(k-1)}``.

``P`` is a Feistel network on ``m``-bit words with a keyed 16-bit
multiply-xorshift-multiply round function:

* width: ``m0 = max(2, bitlen(n-1))``; below 6 bits it is rounded up to even
  (``m`` = 2, 4 or 6), from 6 bits on ``m = m0`` -- the smallest power-of-two
  domain that holds the pool, so that cycle walking takes fewer than two
  evaluations per draw on average; ``m <= 32``, so a half has at most 16 bits;
* halves: left ``a = floor(m/2)`` bits (high), right ``b = m - a`` bits (low);
  a round replaces the left half, ``(L, R) -> (R, L xor F_r(R))`` with
  ``F_r(R) < 2^|L|``, so the half widths alternate (a, b), (b, a), ... and an
  even round count returns to (a, b) -- the alternating split of FFX / NIST
  FF1 for odd widths;
* round function: with key word ``k_r``, ``km = (k_r >> 16) | 1`` (odd) and
  ``kx = k_r mod 2^16``, all arithmetic mod 2^16:
  ``t = R km + kx;  t ^= t >> 8;  t = t C``, ``C = 0x9E37`` (the leading 16
  bits of the golden-ratio constant 2^32/phi); ``F_r(R)`` is the top ``|L|``
  bits of ``t``.  For every key, ``R -> t`` is a bijection of the 16-bit words
  (an affine map with odd slope, an xorshift and an odd multiplication);
* rounds: 6 for ``m >= 8`` (halves of at least 4 bits), 12 below, where
  halves of 1 to 3 bits mix slowly;
* round keys: ``k_r = w_r`` for ``r < 8`` and ``k_r = w_{r-8} xor 0x9E3779B9``
  for ``r = 8..11``, with ``w`` the eight 32-bit words of the row's Philox
  output.

All operations of a round act on 16-bit words, so two draws fit one 32-bit
register and are advanced by the same packed 16-bit instruction.

Values ``>= n`` are cycle-walked (re-encrypted until they fall in range),
which restricts a permutation of ``[0, 2^m)`` to one of ``[0, n)`` (Black and
Rogaway, "Ciphers with arbitrary finite domains", 2002).

Pinned by: the 16-bit map ``R -> t`` is a bijection for every key (an even
slope would break it); exhaustive bijectivity of the network for every width
up to 16 bits; distinctness and range of cycle-walked draws; chi-square
uniformity over independent keys of inclusion, of the first draw, of the
ordered pair (P(0), P(1)) and of the ordered triple (P(0), P(1), P(2)).  The
particular permutation is a definitional choice (any uniform draw realises the
paper's sampling); the GPU reproduces it bit for bit.
"""

import numpy as np

_M16 = np.uint64(0xFFFF)
MIX_C = np.uint64(0x9E37)
KEY_TWEAK = np.uint64(0x9E3779B9)
WORDS = 8          # row words (round-key material)


def mix16(r, k):
    """The keyed 16-bit mixing map t(R) of one round (before the top bits are
    taken): uint64 arrays, r < 2^16, k a 32-bit key word."""
    r = np.asarray(r, dtype=np.uint64)
    k = np.asarray(k, dtype=np.uint64)
    km = ((k >> np.uint64(16)) & _M16) | np.uint64(1)
    kx = k & _M16
    t = (r * km + kx) & _M16
    t = t ^ (t >> np.uint64(8))
    return (t * MIX_C) & _M16


def round_fn(r, k, width):
    """F_r(R): the top ``width`` bits (1..16) of mix16(R, k_r)."""
    return mix16(r, k) >> np.uint64(16 - width)


def domain_bits(n):
    """Word width m for pool sizes n (elementwise): max(2, bitlen(n-1)),
    rounded up to even below 6.  n = 1 gives 2 (unused: P is 0 there)."""
    n = np.asarray(n, dtype=np.int64)
    m = np.zeros(n.shape, dtype=np.int64)
    v = np.maximum(n - 1, 0)
    while (v > 0).any():          # bit length of n - 1
        m += (v > 0)
        v >>= 1
    m = np.maximum(m, 2)
    return np.where(m < 6, m + (m & 1), m)


def rounds(m):
    """Round count for width m (a scalar)."""
    return 6 if m >= 8 else 12


def round_key(w, r):
    """k_r from the row words w (..., 8)."""
    return w[..., r] if r < WORDS else (w[..., r - WORDS] ^ KEY_TWEAK)


def feistel(x, w, m):
    """One application of the keyed permutation of [0, 2^m) for one width m.

    x: uint64 array of values < 2^m.  w: uint64 array (..., 8) of row words
    with leading shape equal to x's.  m: a scalar width from domain_bits.
    """
    assert 2 <= m <= 32, m
    x = np.asarray(x, dtype=np.uint64)
    a = m // 2
    b = m - a
    left = x >> np.uint64(b)
    right = x & np.uint64((1 << b) - 1)
    wl, wr = a, b
    for r in range(rounds(m)):
        f = round_fn(right, round_key(w, r), wl)
        left, right = right, left ^ f
        wl, wr = wr, wl
    return (left << np.uint64(wr)) | right


def _feistel_by_width(x, w, m):
    """feistel over arrays whose widths m differ element by element."""
    out = np.empty_like(x)
    for mm in np.unique(m):
        sel = m == mm
        out[sel] = feistel(x[sel], w[sel], int(mm))
    return out


def permute(j, w, n):
    """P(j) for the keyed permutation of [0, n), by cycle walking.

    j: uint64 array of values < n.  w: row words (j.shape + (8,)) or one word
    set (8,).  n: pool sizes >= 1, broadcast with j.
    """
    j = np.asarray(j, dtype=np.uint64)
    n = np.broadcast_to(np.asarray(n, dtype=np.uint64), j.shape)
    w = np.broadcast_to(np.asarray(w, dtype=np.uint64), j.shape + (WORDS,))
    m = domain_bits(n.astype(np.int64))
    x = _feistel_by_width(j, w, m)
    bad = x >= n
    while bad.any():
        x[bad] = _feistel_by_width(x[bad], w[bad], m[bad])
        bad = x >= n
    return np.where(n == np.uint64(1), np.uint64(0), x)


def draw(k, n, w):
    """The k keys {P(0), ..., P(k-1)} drawn from [0, n) (distinct, unsorted)."""
    if k <= 0 or n <= 0:
        return np.zeros(0, dtype=np.uint64)
    return permute(np.arange(k, dtype=np.uint64), np.asarray(w, dtype=np.uint64), n)
