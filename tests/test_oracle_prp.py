"""Pins for the oracle's exact-k draw (see oracle/prp.py)."""
import numpy as np
import pytest
from scipy.stats import chi2

from oracle import prp


def test_round_mixer_is_a_bijection_of_16_bit_words():
    """For every key the 16-bit map of a round (affine with odd slope,
    xorshift, odd multiplication) permutes [0, 2^16); a slope that lost its
    forced low bit would collapse half the words."""
    rng = np.random.default_rng(1)
    r = np.arange(1 << 16, dtype=np.uint64)
    keys = np.concatenate([[0, 1, 0xFFFF, 0x10000, 0xFFFFFFFF, 0x9E3779B9],
                           rng.integers(0, 2**32, size=40, dtype=np.uint64)])
    for k in keys:
        t = prp.mix16(r, np.uint64(k))
        assert t.max() < (1 << 16)
        assert np.unique(t).size == (1 << 16), hex(int(k))
    # the same map with an even slope (the low bit of the high key half
    # cleared) is not one: the pin above can fail
    even = ((r * np.uint64(0x9E36)) & np.uint64(0xFFFF))
    assert np.unique(even).size < (1 << 16)


def test_round_function_takes_the_top_bits():
    rng = np.random.default_rng(2)
    r = rng.integers(0, 1 << 16, size=500, dtype=np.uint64)
    k = rng.integers(0, 2**32, size=500, dtype=np.uint64)
    t = prp.mix16(r, k)
    for w in range(1, 17):
        f = prp.round_fn(r, k, w)
        assert f.max() < (1 << w)
        assert np.array_equal(f, t >> np.uint64(16 - w))


def test_domain_bits_and_rounds():
    ns = [1, 2, 3, 4, 5, 8, 9, 16, 17, 32, 33, 64, 65, 4096, 4097, 65536, 65537, 262144]
    want = [2, 2, 2, 2, 4, 4, 4, 4, 6, 6, 6, 6, 7, 12, 13, 16, 17, 18]
    assert list(prp.domain_bits(np.array(ns))) == want
    assert [prp.rounds(m) for m in (2, 4, 6, 7, 8, 18, 32)] == [12, 12, 12, 12, 6, 6, 6]
    # the domain never exceeds twice the pool once the width is exact (n > 32)
    for n in [33, 100, 1000, 65536, 65537, 262144]:
        assert (1 << int(prp.domain_bits(n))) < 2 * n


def test_feistel_matches_a_plain_python_rewrite():
    """The vectorised rounds equal a scalar rewrite of the stated network
    (a consistency check of the vectorisation, not a pin)."""
    rng = np.random.default_rng(7)

    def F(right, k, width):
        km, kx = (k >> 16) | 1, k & 0xFFFF
        t = (right * km + kx) & 0xFFFF
        t ^= t >> 8
        t = (t * 0x9E37) & 0xFFFF
        return t >> (16 - width)

    for m in [2, 4, 6, 7, 8, 9, 16, 17, 31, 32]:
        w = [int(v) for v in rng.integers(0, 2**32, size=8, dtype=np.uint64)]
        xs = rng.integers(0, 1 << m, size=40, dtype=np.uint64)
        got = prp.feistel(xs, np.broadcast_to(np.array(w, dtype=np.uint64), (40, 8)), m)
        a, b = m // 2, m - m // 2
        for x, g in zip(xs, got):
            left, right, wl = int(x) >> b, int(x) & ((1 << b) - 1), a
            for r in range(12 if m < 8 else 6):
                k = w[r] if r < 8 else w[r - 8] ^ 0x9E3779B9
                left, right = right, left ^ F(right, k, wl)
                wl = b if wl == a and r % 2 == 0 else a
            assert ((left << b) | right) == int(g)


@pytest.mark.parametrize("m", [2, 4, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15, 16])
def test_feistel_is_a_bijection(m):
    rng = np.random.default_rng(m)
    for _ in range(2 if m >= 15 else 4):
        w = rng.integers(0, 2**32, size=8, dtype=np.uint64)
        x = np.arange(1 << m, dtype=np.uint64)
        y = prp.feistel(x, np.broadcast_to(w, x.shape + (8,)), m)
        assert y.max() < (1 << m)
        assert np.unique(y).size == (1 << m)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 7, 17, 33, 100, 257, 1000, 4097, 40000])
def test_cycle_walk_permutes_the_pool(n):
    rng = np.random.default_rng(n)
    w = rng.integers(0, 2**32, size=8, dtype=np.uint64)
    y = prp.permute(np.arange(n, dtype=np.uint64), w, n)
    assert np.array_equal(np.sort(y), np.arange(n, dtype=np.uint64))


def test_draw_is_distinct_and_in_range():
    rng = np.random.default_rng(3)
    for n in [1, 2, 9, 333, 5000]:
        for k in [1, n // 3 + 1, n]:
            w = rng.integers(0, 2**32, size=8, dtype=np.uint64)
            d = prp.draw(k, n, w)
            assert d.size == k and np.unique(d).size == k and d.max() < n


def _draws(n, k, trials, seed):
    keys = np.random.default_rng(seed).integers(0, 2**32, size=(trials, 8), dtype=np.uint64)
    j = np.tile(np.arange(k, dtype=np.uint64), trials)
    return prp.permute(j, np.repeat(keys, k, axis=0), n).astype(np.int64).reshape(trials, k)


def _chi2_ok(obs, expect, df):
    stat = float(((obs - expect) ** 2 / expect).sum())
    return stat < chi2.ppf(1 - 1e-4, df), stat


@pytest.mark.parametrize("n,k", [(5, 2), (7, 3), (13, 1), (33, 10), (65, 6), (300, 20)])
def test_inclusion_and_first_draw_are_uniform(n, k):
    """Over many independent keys each pool element is drawn with
    probability k/n, and the first drawn key is uniform (chi-square, 1e-4
    false-alarm level)."""
    trials = 20000
    x = _draws(n, k, trials, n * 100 + k)
    ok, stat = _chi2_ok(np.bincount(x.ravel(), minlength=n), trials * k / n, n - 1)
    assert ok, stat
    ok, stat = _chi2_ok(np.bincount(x[:, 0], minlength=n), trials / n, n - 1)
    assert ok, stat


@pytest.mark.parametrize("n", [4, 5, 7, 9, 16, 17, 32, 33, 65, 129, 257])
def test_successive_draws_are_jointly_uniform(n):
    """(P(0), P(1)) is uniform over ordered pairs of distinct keys, one pair
    per independent key (so the cells are a true multinomial); widths with
    1- and 2-bit halves (n <= 16) included."""
    trials = max(40000, 25 * n * (n - 1))
    x = _draws(n, 2, trials, 1000 + n)
    counts = np.bincount(x[:, 0] * n + x[:, 1], minlength=n * n).reshape(n, n)
    off = ~np.eye(n, dtype=bool)
    assert counts[~off].sum() == 0
    ok, stat = _chi2_ok(counts[off], trials / (n * (n - 1)), n * (n - 1) - 1)
    assert ok, stat


@pytest.mark.parametrize("n", [5, 9, 17, 33])
def test_three_successive_draws_are_jointly_uniform(n):
    """(P(0), P(1), P(2)) is uniform over ordered triples of distinct keys,
    one triple per independent key (12-round widths)."""
    trials = 25 * n * (n - 1) * (n - 2)
    x = _draws(n, 3, trials, 2000 + n)
    cell = (x[:, 0] * n + x[:, 1]) * n + x[:, 2]
    counts = np.bincount(cell, minlength=n ** 3)
    i = np.arange(n ** 3)
    a, b, c = i // (n * n), (i // n) % n, i % n
    distinct = (a != b) & (b != c) & (a != c)
    assert counts[~distinct].sum() == 0
    ok, stat = _chi2_ok(counts[distinct], trials / distinct.sum(), int(distinct.sum()) - 1)
    assert ok, stat


@pytest.mark.parametrize("n", [300, 4097, 65537, 262144])
def test_draws_on_large_pools_are_jointly_uniform_in_bins(n):
    """On six-round widths: (P(j), P(j+1)) for j = 0 and 7 in 32 x 32 bins,
    and (P(0), P(1), P(2)) in 16^3 bins, over independent keys."""
    rng = np.random.default_rng(3000 + n)
    trials = 100000
    for j0 in (0, 7):
        keys = rng.integers(0, 2**32, size=(trials, 8), dtype=np.uint64)
        j = np.tile(np.array([j0, j0 + 1], dtype=np.uint64), trials)
        x = prp.permute(j, np.repeat(keys, 2, axis=0), n).astype(np.int64).reshape(trials, 2)
        bins = x * 32 // n
        # bin masses: equal up to the pool not dividing into 32 bins
        mass = np.bincount(np.arange(n) * 32 // n, minlength=32) / n
        expect = trials * np.outer(mass, mass).ravel()
        ok, stat = _chi2_ok(np.bincount(bins[:, 0] * 32 + bins[:, 1], minlength=1024), expect, 1023)
        assert ok, (j0, stat)
    x = _draws(n, 3, 200000, 4000 + n)
    bins = x * 16 // n
    mass = np.bincount(np.arange(n) * 16 // n, minlength=16) / n
    expect = 200000 * np.einsum("i,j,k->ijk", mass, mass, mass).ravel()
    cell = (bins[:, 0] * 16 + bins[:, 1]) * 16 + bins[:, 2]
    ok, stat = _chi2_ok(np.bincount(cell, minlength=4096), expect, 4095)
    assert ok, stat


def test_walk_needs_fewer_than_two_evaluations_per_draw():
    """With a power-of-two domain below twice the pool the cycle walk averages
    fewer than two permutation evaluations per draw."""
    rng = np.random.default_rng(11)
    for n in [33, 600, 5000, 40000, 65537]:
        w = rng.integers(0, 2**32, size=8, dtype=np.uint64)
        m = int(prp.domain_bits(n))
        x = np.arange(n, dtype=np.uint64)
        steps = np.ones(n)
        y = prp.feistel(x, np.broadcast_to(w, (n, 8)), m)
        while (y >= n).any():
            bad = y >= n
            steps[bad] += 1
            y[bad] = prp.feistel(y[bad], np.broadcast_to(w, (int(bad.sum()), 8)), m)
        assert steps.mean() < 2.0


def _subset_counts(n, k, trials, seed):
    """How often each k-subset of [0, n) is the drawn set, over independent
    keys (one draw per key, so the cells are a true multinomial)."""
    from math import comb
    x = _draws(n, k, trials, seed)
    if n <= 62:
        code = (np.int64(1) << x).sum(axis=1)
    else:                                   # k = 2 on a larger pool
        xs = np.sort(x, axis=1)
        code = xs[:, 0] * n + xs[:, 1]
    _, c = np.unique(code, return_counts=True)
    obs = np.zeros(comb(n, k))
    obs[:c.size] = c
    return obs


SUBSET_CASES = [(6, 3), (8, 4), (10, 5), (12, 6), (16, 4), (20, 3), (33, 2), (33, 3), (130, 2)]


@pytest.mark.parametrize("n,k", SUBSET_CASES)
def test_drawn_subsets_are_uniform(n, k):
    """The reading of the paper's per-seed draw is an exact-k uniform draw
    without replacement: every k-subset of the pool equally likely.  Tested
    directly over all C(n, k) subsets (chi-square at the 1e-4 false-alarm
    level), on 12-round widths and on a 6-round one (n = 130)."""
    from math import comb
    C = comb(n, k)
    trials = max(30000, 40 * C)
    obs = _subset_counts(n, k, trials, 5000 + n * 7 + k)
    assert obs.sum() == trials
    ok, stat = _chi2_ok(obs, trials / C, C - 1)
    assert ok, stat


@pytest.mark.parametrize("n,k,rounds", [(6, 3, 2), (8, 4, 2), (12, 6, 4), (16, 4, 4), (20, 3, 4),
                                        (33, 2, 4), (130, 2, 2), (8, 4, 6), (12, 6, 6)])
def test_the_subset_test_rejects_weaker_networks(monkeypatch, n, k, rounds):
    """The subset test has the power to catch a weaker mix: the same network
    with fewer rounds fails it -- 2 or 4 rounds anywhere, and 6 rounds on
    the smallest pools, which is why pools below 8 bits take 12."""
    from math import comb
    monkeypatch.setattr(prp, "rounds", lambda m: rounds)
    C = comb(n, k)
    trials = max(30000, 40 * C)
    obs = _subset_counts(n, k, trials, 5000 + n * 7 + k)
    ok, stat = _chi2_ok(obs, trials / C, C - 1)
    assert not ok, stat
