"""Pins for the oracle's Philox4x64-10 (see oracle/philox.py).

numpy.random.Philox is an independent implementation of the same published
generator (Salmon et al., SC'11).  It increments its 256-bit counter before
producing a block, so block(c) is numpy's first output for counter c - 1.
"""
import numpy as np
import pytest

from oracle import philox


def numpy_block(counter, key):
    c = sum(int(w) << (64 * i) for i, w in enumerate(counter))
    c = (c - 1) % (1 << 256)
    words = np.array([(c >> (64 * i)) & (2**64 - 1) for i in range(4)], dtype=np.uint64)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=words)
    return [int(x) for x in bg.random_raw(4)]


def test_mulhilo_against_python_ints():
    rng = np.random.default_rng(5)
    a = rng.integers(0, 2**64, size=1000, dtype=np.uint64)
    b = rng.integers(0, 2**64, size=1000, dtype=np.uint64)
    hi, lo = philox.mulhilo64(a, b)
    for x, y, h, l in zip(a[:200], b[:200], hi[:200], lo[:200]):
        p = int(x) * int(y)
        assert int(h) == p >> 64 and int(l) == p & (2**64 - 1)
    top = np.uint64(2**64 - 1)
    h, l = philox.mulhilo64(top, top)
    assert int(h) == (2**64 - 1) ** 2 >> 64 and int(l) == 1


@pytest.mark.parametrize("case", range(40))
def test_block_matches_numpy(case):
    rng = np.random.default_rng(100 + case)
    if case == 0:
        ctr, key = [0, 0, 0, 0], [0, 0]          # borrow through all words
    elif case == 1:
        ctr, key = [2**64 - 1] * 4, [2**64 - 1] * 2
    else:
        ctr = [int(x) for x in rng.integers(0, 2**64, size=4, dtype=np.uint64)]
        key = [int(x) for x in rng.integers(0, 2**64, size=2, dtype=np.uint64)]
        if case % 3 == 0:
            ctr[0] = 0                            # exercise the borrow
    got = philox.philox4x64_10([np.uint64(c) for c in ctr], [np.uint64(k) for k in key])
    assert [int(g) for g in got] == numpy_block(ctr, key)


def test_row_round_keys_layout():
    """Eight row words = the four 64-bit outputs split low half first,
    for key (seed, 0) and counter (q, kv_head, layer, 0); vectorised calls agree
    with scalar ones."""
    seeds = np.array([0, 1, 69, 2**40 + 3], dtype=np.uint64)
    qs = np.array([0, 1, 511, 65535], dtype=np.uint64)
    rk = philox.row_round_keys(seeds[None, :], qs[:, None], np.uint64(1), np.uint64(7))
    assert rk.shape == (4, 4, 8)
    for a, q in enumerate(qs):
        for b, s in enumerate(seeds):
            out = numpy_block([int(q), 1, 7, 0], [int(s), 0])
            words = []
            for w in out:
                words += [w & 0xFFFFFFFF, w >> 32]
            assert [int(x) for x in rk[a, b]] == words
