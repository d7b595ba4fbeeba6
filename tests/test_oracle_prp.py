"""Pins for the oracle's exact-k draw (see oracle/prp.py)."""
import numpy as np
import pytest
from sklearn.utils import murmurhash3_32

from oracle import prp


def test_fmix32_against_sklearn_murmurhash3():
    """MurmurHash3_x86_32 of the empty string with seed x is fmix32(x)."""
    rng = np.random.default_rng(1)
    xs = np.concatenate([[0, 1, 2, 0xFFFFFFFF, 0x80000000],
                         rng.integers(0, 2**32, size=3000, dtype=np.uint64)])
    got = prp.fmix32(xs.astype(np.uint64))
    want = np.array([murmurhash3_32(b"", seed=int(x), positive=True) for x in xs], dtype=np.uint64)
    assert np.array_equal(got, want)
    assert int(prp.fmix32(np.uint64(1))) == 0x514E28B7   # published test vector


def test_domain_bits():
    ns = [1, 2, 3, 4, 5, 8, 9, 16, 17, 64, 65, 4096, 4097, 65536, 65537]
    want = [2, 2, 2, 2, 4, 4, 4, 4, 6, 6, 8, 12, 14, 16, 18]
    assert list(prp.domain_bits(np.array(ns))) == want


@pytest.mark.parametrize("m", [2, 4, 6, 8, 10, 12, 14, 16])
def test_feistel_is_a_bijection(m):
    rng = np.random.default_rng(m)
    for _ in range(2 if m == 16 else 4):
        rk = rng.integers(0, 2**32, size=6, dtype=np.uint64)
        x = np.arange(1 << m, dtype=np.uint64)
        y = prp.feistel(x, np.broadcast_to(rk, x.shape + (6,)), m)
        assert y.max() < (1 << m)
        assert np.unique(y).size == (1 << m)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 7, 17, 100, 257, 1000, 4097, 40000])
def test_cycle_walk_permutes_the_pool(n):
    rng = np.random.default_rng(n)
    rk = rng.integers(0, 2**32, size=6, dtype=np.uint64)
    y = prp.permute(np.arange(n, dtype=np.uint64), rk, n)
    assert np.array_equal(np.sort(y), np.arange(n, dtype=np.uint64))


def test_draw_is_distinct_and_in_range():
    rng = np.random.default_rng(3)
    for n in [1, 2, 9, 333, 5000]:
        for k in [1, n // 3 + 1, n]:
            rk = rng.integers(0, 2**32, size=6, dtype=np.uint64)
            d = prp.draw(k, n, rk)
            assert d.size == k and np.unique(d).size == k and d.max() < n


@pytest.mark.parametrize("n,k", [(7, 3), (13, 1), (33, 10)])
def test_inclusion_is_uniform(n, k):
    """Over many independent keys each pool element is drawn with
    probability k/n (chi-square, 1e-4 false-alarm level)."""
    from scipy.stats import chi2
    rng = np.random.default_rng(n * 100 + k)
    trials = 6000
    keys = rng.integers(0, 2**32, size=(trials, 6), dtype=np.uint64)
    j = np.tile(np.arange(k, dtype=np.uint64), trials)
    x = prp.permute(j, np.repeat(keys, k, axis=0), n)
    counts = np.bincount(x.astype(np.int64), minlength=n)
    expect = trials * k / n
    stat = float(((counts - expect) ** 2 / expect).sum())
    assert stat < chi2.ppf(1 - 1e-4, n - 1)
    # the first drawn key is uniform as well (no bias toward small values)
    first = x.reshape(trials, k)[:, 0].astype(np.int64)
    c1 = np.bincount(first, minlength=n)
    e1 = trials / n
    assert float(((c1 - e1) ** 2 / e1).sum()) < chi2.ppf(1 - 1e-4, n - 1)
