"""Pins for the oracle's sparse attention (see oracle/attention.py)."""
import numpy as np
import pytest
import torch

from oracle import attention as att
from oracle import geometry as geo
from synth import gaussian_qkv


def spec(**kw):
    base = dict(mode=geo.STOCHASTIC, density_ppm=100_000, seed=0, n_seeds=1, layer=0,
                N=64, heads=1, causal=1, block=0)
    base.update(kw)
    return geo.MaskSpec(**base)


@pytest.mark.parametrize("mode", [geo.STOCHASTIC, geo.STRUCTURAL])
def test_full_density_equals_dense_causal_attention(mode):
    """At 100% density the sets are the causal triangle, so RIS attention is
    dense causal softmax attention (the "Full Dense Baseline 100%" row of the
    32k results table).  Checked against a textbook numpy version and against
    torch's scaled_dot_product_attention on the CPU."""
    Hq, Hkv, N, D = 6, 2, 96, 64
    Q, K, V = gaussian_qkv(Hq, Hkv, N, D, seed=3)
    sp = spec(mode=mode, density_ppm=10**6, N=N, heads=Hkv, n_seeds=2, block=16)
    row_ptr, col_idx = geo.build_csr(sp)
    got = att.sparse_attention(Q, K, V, row_ptr, col_idx)
    np.testing.assert_allclose(got, att.dense_causal(Q, K, V), rtol=0, atol=1e-12)
    G = Hq // Hkv
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q.astype(np.float64))[None],
        torch.from_numpy(np.repeat(K, G, axis=0).astype(np.float64))[None],
        torch.from_numpy(np.repeat(V, G, axis=0).astype(np.float64))[None],
        is_causal=True)[0].numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("mode,ppm,S", [(geo.STOCHASTIC, 150_000, 3), (geo.STRUCTURAL, 120_000, 2)])
def test_brute_force_boolean_mask(mode, ppm, S):
    """Tiny N: materialise the N x N boolean mask of each KV head from the
    plain per-row definition and run masked dense softmax (-inf fill)."""
    Hq, Hkv, N, D = 4, 2, 80, 32
    Q, K, V = gaussian_qkv(Hq, Hkv, N, D, seed=4)
    sp = spec(mode=mode, density_ppm=ppm, N=N, heads=Hkv, n_seeds=S, block=16, seed=7)
    row_ptr, col_idx = geo.build_csr(sp)
    got = att.sparse_attention(Q, K, V, row_ptr, col_idx)
    G = Hq // Hkv
    for h in range(Hq):
        g = h // G
        mask = np.zeros((N, N), dtype=bool)
        for q in range(N):
            mask[q, geo.row_set(sp, g, q)] = True
        s = (Q[h].astype(np.float64) @ K[g].astype(np.float64).T) / np.sqrt(D)
        s = np.where(mask, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        np.testing.assert_allclose(got[h], p @ V[g].astype(np.float64), rtol=0, atol=1e-12)


def test_weights_sum_to_one_and_vanish_off_the_set():
    """With V = identity (one-hot per key) the output row is p itself."""
    N = D = 64
    Q, K, _ = gaussian_qkv(1, 1, N, D, seed=5)
    V = np.eye(N, dtype=np.float32)[None]
    sp = spec(density_ppm=200_000, N=N, n_seeds=2)
    row_ptr, col_idx = geo.build_csr(sp)
    P = att.sparse_attention(Q, K, V, row_ptr, col_idx)[0]
    np.testing.assert_allclose(P.sum(axis=1), 1.0, rtol=0, atol=1e-13)
    for q in range(N):
        off = np.setdiff1d(np.arange(N), col_idx[row_ptr[q]:row_ptr[q + 1]])
        assert np.all(P[q, off] == 0.0)
        assert np.all(P[q, col_idx[row_ptr[q]:row_ptr[q + 1]]] > 0.0)


def test_pfus_is_one_softmax_over_the_set_union():
    """Heavy seed overlap (d = 50%, 8 seeds): the result is one softmax over
    the *set* union, and differs from (a) a softmax over the multiset of all
    seeds' draws (duplicates counted) and (b) the average of per-seed
    normalised outputs -- the post-combination the paper rejects."""
    N, D = 48, 16
    Q, K, V = gaussian_qkv(1, 1, N, D, seed=6)
    sp = spec(density_ppm=500_000, N=N, n_seeds=8)
    row_ptr, col_idx = geo.build_csr(sp)
    got = att.sparse_attention(Q, K, V, row_ptr, col_idx)[0]
    scale = 1 / np.sqrt(D)
    diff_multi, diff_post = [], []
    for q in range(8, N):
        u = geo.row_set(sp, 0, q)
        np.testing.assert_allclose(got[q], att.attend_one(Q[0, q], K[0, u], V[0, u], scale), atol=1e-13)
        draws = [geo.seed_draws(sp, 0, q, s) for s in range(8)]
        multi = np.concatenate(draws)
        assert multi.size > u.size                        # overlap exists
        diff_multi.append(np.abs(att.attend_one(Q[0, q], K[0, multi], V[0, multi], scale) - got[q]).max())
        post = np.mean([att.attend_one(Q[0, q], K[0, d], V[0, d], scale) for d in draws], axis=0)
        diff_post.append(np.abs(post - got[q]).max())
    assert min(diff_multi) > 0 and np.median(diff_multi) > 1e-3
    assert min(diff_post) > 0 and np.median(diff_post) > 1e-3


def test_empty_set_gives_zero_and_single_key_gives_its_value():
    q = np.ones(8)
    assert np.all(att.attend_one(q, np.zeros((0, 8)), np.zeros((0, 8)), 0.3) == 0)
    v = np.arange(8.0)
    np.testing.assert_array_equal(att.attend_one(q, np.ones((1, 8)), v[None], 0.3), v)
