"""Pins for the oracle's Hybrid-Anchor decode step (oracle/decode.py)."""
import numpy as np
import pytest

from oracle import attention as att
from oracle import decode as dec
from oracle import geometry as geo


def spec(**kw):
    base = dict(mode=geo.STOCHASTIC, density_ppm=20_000, seed=3, n_seeds=5, layer=1,
                N=3000, heads=2, causal=1, block=0)
    base.update(kw)
    return geo.MaskSpec(**base)


@pytest.mark.parametrize("mode,block", [(geo.STOCHASTIC, 0), (geo.STRUCTURAL, 64)])
def test_first_step_equals_prefill_row(mode, block):
    """At t = t0 the cached anchor plus window and sink is exactly the full
    prefill geometry's row t0 (window L, anchor A) -- two independent
    constructions of the same set."""
    for L, A in [(1024, 4), (50, 0), (0, 9), (1, 1)]:
        sp = spec(mode=mode, block=block, window=L, anchor=A)
        for g in range(sp.heads):
            for t0 in [0, 1, 63, 64, 999, 2047, 2999]:
                anc = dec.stochastic_anchor(sp, g, t0)
                assert np.array_equal(dec.step_set(anc, t0, L, A), geo.row_set(sp, g, t0))


def test_step_set_against_python_sets():
    """Brute force with Python set algebra over a run of decode steps."""
    rng = np.random.default_rng(0)
    anchor = np.unique(rng.integers(0, 500, size=60))
    for t in range(500, 700, 7):
        for L, A in [(0, 0), (1, 0), (16, 3), (300, 600), (1000, 1)]:
            want = set(int(x) for x in anchor if x <= t)
            want |= {t - i for i in range(L) if t - i >= 0}
            want |= {i for i in range(A) if i <= t}
            got = dec.step_set(anchor, t, L, A)
            assert list(got) == sorted(want)
            assert len(np.unique(got)) == len(got)


def test_window_and_sink_shapes():
    """With no anchor the set is exactly the window (L keys ending at t) and
    the sink (the first A tokens); the anchor only ever adds keys."""
    for t in [0, 5, 100, 5000]:
        w = dec.step_set(np.zeros(0, np.int64), t, 64, 0)
        assert len(w) == min(64, t + 1) and w[-1] == t and np.all(np.diff(w) == 1)
        s = dec.step_set(np.zeros(0, np.int64), t, 0, 10)
        assert np.array_equal(s, np.arange(min(10, t + 1)))
        full = dec.step_set(np.arange(t + 1), t, 64, 10)
        assert np.array_equal(full, np.arange(t + 1))


def test_anchor_is_frozen_between_window_and_sink():
    """Later steps change only the window: the part of the set between the
    sink and the window is the anchor's, whatever t is."""
    sp = spec(window=128, anchor=4)
    t0 = 1500
    anc = dec.stochastic_anchor(sp, 1, t0)
    for t in [t0, t0 + 1, t0 + 200, t0 + 1000]:
        s = dec.step_set(anc, t, 128, 4)
        lo, hi = 4, t - 128 + 1
        assert np.array_equal(s[(s >= lo) & (s < hi)], anc[(anc >= lo) & (anc < hi)])
        assert s[-1] == t


def test_anchor_does_not_depend_on_sequence_capacity():
    """The anchor is a function of (seed, layer, head, t0) only."""
    a = dec.stochastic_anchor(spec(N=1001), 0, 1000)
    b = dec.stochastic_anchor(spec(N=3000), 0, 1000)
    assert np.array_equal(a, b)
    with pytest.raises(ValueError):
        dec.stochastic_anchor(spec(N=1000), 0, 1000)


def test_decode_attention_full_set_is_dense_causal_last_row():
    rng = np.random.default_rng(1)
    G, T, D = 3, 40, 16
    q = rng.standard_normal((G, D))
    K = rng.standard_normal((T, D))
    V = rng.standard_normal((T, D))
    out = dec.decode_attention(q, K, V, np.arange(T), 1 / np.sqrt(D))
    Qf = np.zeros((G, T, D))
    Qf[:, T - 1] = q
    dense = att.dense_causal(Qf, np.repeat(K[None], G, 0), np.repeat(V[None], G, 0))
    assert np.allclose(out, dense[:, T - 1], atol=1e-12)


def test_decode_attention_is_a_set_function():
    """Order does not matter, a duplicate would (hence the unique merge),
    and the empty set gives zeros."""
    rng = np.random.default_rng(2)
    q = rng.standard_normal((2, 8))
    K = rng.standard_normal((30, 8))
    V = rng.standard_normal((30, 8))
    idx = np.array([0, 3, 7, 12, 29])
    a = dec.decode_attention(q, K, V, idx, 0.5)
    b = dec.decode_attention(q, K, V, idx[::-1], 0.5)
    c = dec.decode_attention(q, K, V, np.append(idx, 7), 0.5)
    assert np.allclose(a, b, atol=1e-14)
    assert not np.allclose(a, c, atol=1e-6)
    assert np.all(dec.decode_attention(q, K, V, idx[:0], 0.5) == 0)
