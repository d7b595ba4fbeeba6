"""Pins for the oracle's geometry (see oracle/geometry.py)."""
import os

import numpy as np
import pytest

from oracle import geometry as geo

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([float(x) for x in line.split()])
    return rows


def spec(**kw):
    base = dict(mode=geo.STOCHASTIC, density_ppm=10_000, seed=0, n_seeds=1, layer=0,
                N=512, heads=1, causal=1, block=0)
    base.update(kw)
    return geo.MaskSpec(**base)


def test_count_rule_reproduces_paper_bmax_table():
    """round-half-up of d * N on N = 65,536 gives every printed B_max."""
    for dens_pct, bmax in _golden("sweet_spot_bmax.txt"):
        ppm = int(round(dens_pct * 10_000))
        assert int(geo.row_count(ppm, 65536)) == int(bmax)
    # ceiling and floor would each miss at least one printed value
    ppm = np.array([int(round(r[0] * 10_000)) for r in _golden("sweet_spot_bmax.txt")])
    want = np.array([int(r[1]) for r in _golden("sweet_spot_bmax.txt")])
    assert not np.array_equal(-(-ppm * 65536 // 10**6), want)
    assert not np.array_equal(ppm * 65536 // 10**6, want)


def test_count_rule_edges():
    n = np.arange(1, 2000)
    assert np.all(geo.row_count(1, n) == 1)                  # never empty
    assert np.array_equal(geo.row_count(10**6, n), n)       # 100% = whole pool
    k = geo.row_count(250_000, n)
    assert np.all((k >= 1) & (k <= n))


def test_paper_block_rule():
    """B = min(0.1 N, B_max): 655 at 64k/1%, 328 at 32k/1%, 3277 at 64k/5%."""
    assert geo.block_size(spec(mode=1, N=65536, density_ppm=10_000)) == 655
    assert geo.block_size(spec(mode=1, N=32768, density_ppm=10_000)) == 328
    assert geo.block_size(spec(mode=1, N=65536, density_ppm=50_000)) == 3277
    assert geo.block_size(spec(mode=1, N=100, density_ppm=10**6)) == 10   # 0.1 N caps
    assert geo.block_size(spec(mode=1, N=65536, block=64)) == 64


def check_csr(sp, row_ptr, col_idx):
    assert row_ptr[0] == 0 and np.all(np.diff(row_ptr) >= 1)
    assert row_ptr[-1] == col_idx.size
    for r in range(sp.heads * sp.N):
        q = r % sp.N
        row = col_idx[row_ptr[r]:row_ptr[r + 1]].astype(np.int64)
        assert np.all(np.diff(row) > 0)                    # ascending, unique
        assert row[0] >= 0
        assert row[-1] <= (q if sp.causal else sp.N - 1)   # causal


def test_tiny_workload_total_and_counts():
    """Single seed: every row holds exactly k(q) keys; the 512-token, 10%
    workload therefore holds sum_q k(q) = 13,162 pairs."""
    sp = spec(density_ppm=100_000, N=512)
    row_ptr, col_idx = geo.build_csr(sp)
    check_csr(sp, row_ptr, col_idx)
    counts = np.diff(row_ptr)
    assert np.array_equal(counts, geo.row_count(100_000, np.arange(1, 513)))
    assert row_ptr[-1] == 13_162


def test_structural_single_seed_counts_and_clique_suffix():
    sp = spec(mode=geo.STRUCTURAL, density_ppm=50_000, N=700, block=64, heads=2, n_seeds=1)
    row_ptr, col_idx = geo.build_csr(sp)
    check_csr(sp, row_ptr, col_idx)
    for h in range(2):
        for q in range(sp.N):
            r = h * sp.N + q
            row = col_idx[row_ptr[r]:row_ptr[r + 1]]
            start = (q // 64) * 64
            clique = q - start + 1
            k = int(geo.row_count(50_000, q + 1))
            kg = min(start, max(0, k - clique))
            assert row.size == clique + kg
            assert np.array_equal(row[-clique:], np.arange(start, q + 1))   # suffix
            assert np.all(row[:kg] < start)


def test_full_density_is_the_causal_triangle():
    for mode in (geo.STOCHASTIC, geo.STRUCTURAL):
        sp = spec(mode=mode, density_ppm=10**6, N=300, n_seeds=3, block=32)
        row_ptr, col_idx = geo.build_csr(sp)
        for q in range(sp.N):
            assert np.array_equal(col_idx[row_ptr[q]:row_ptr[q + 1]], np.arange(q + 1))


def test_noncausal_pool_is_whole_sequence():
    sp = spec(causal=0, density_ppm=200_000, N=257, n_seeds=2)
    row_ptr, col_idx = geo.build_csr(sp)
    check_csr(sp, row_ptr, col_idx)
    assert col_idx.max() > 200    # early rows see late keys


@pytest.mark.parametrize("mode", [geo.STOCHASTIC, geo.STRUCTURAL])
def test_vectorised_rows_equal_plain_definition(mode):
    sp = spec(mode=mode, density_ppm=37_000, N=3000, n_seeds=5, heads=2, block=50, layer=3, seed=11)
    qs = np.array([0, 1, 2, 49, 50, 51, 999, 1777, 2998, 2999])
    for h in range(2):
        fast = geo.row_sets(sp, h, qs)
        for q, f in zip(qs, fast):
            assert np.array_equal(f, geo.row_set(sp, h, int(q)))


def test_layers_heads_and_seeds_change_the_sets():
    sp = spec(density_ppm=50_000, N=2000, n_seeds=2, heads=2)
    q = 1999
    a = geo.row_set(sp, 0, q)
    assert not np.array_equal(a, geo.row_set(sp, 1, q))
    assert not np.array_equal(a, geo.row_set(geo.MaskSpec(**{**sp.__dict__, "layer": 1}), 0, q))
    assert not np.array_equal(a, geo.row_set(geo.MaskSpec(**{**sp.__dict__, "seed": 5}), 0, q))


def test_union_coverage_matches_paper_equation():
    """Union fraction of S exact-k draws at density d tends to
    U = 1 - (1 - d)^S; the paper prints 50.5% (d = 1%) and 97.2% (d = 5%)
    at 70 seeds."""
    for d, S, u_pct in _golden("union_coverage.txt"):
        u = 1.0 - (1.0 - d) ** S
        assert abs(100 * u - u_pct) < 0.05            # the printed rounding
        sp = spec(density_ppm=int(round(d * 1e6)), N=10_000, n_seeds=int(S), causal=0)
        qs = np.arange(0, 24)
        fracs = [s.size / 10_000 for s in geo.row_sets(sp, 0, qs)]
        # std of one row's fraction <= sqrt(U(1-U)/n) ~ 0.005; mean of 24 rows
        assert abs(np.mean(fracs) - u) < 0.004


def test_capture_probability_of_repeated_term():
    """A term present at k positions is captured by at least one of S seeds
    at density rho with probability about 1 - (1 - rho)^(k S) (Methods,
    "Ensemble Stochastic Projection and Retrieval Coverage")."""
    N, rho, S, k = 5000, 0.01, 10, 3
    sp = spec(density_ppm=int(rho * 1e6), N=N, n_seeds=S, causal=0)
    term = np.array([123, 2222, 4321])
    rows = geo.row_sets(sp, 0, np.arange(0, 1500))
    hit = np.mean([np.isin(term, r).any() for r in rows])
    want = 1 - (1 - rho) ** (k * S)
    assert abs(hit - want) < 0.035                 # ~3 sigma over 1500 rows


def test_nnz_bound_is_an_upper_bound():
    for mode in (geo.STOCHASTIC, geo.STRUCTURAL):
        sp = spec(mode=mode, density_ppm=80_000, N=900, n_seeds=4, heads=2, block=40)
        row_ptr, _ = geo.build_csr(sp)
        assert geo.nnz_upper_bound(sp) >= row_ptr[-1]
    sp = spec(density_ppm=100_000, N=512)
    assert geo.nnz_upper_bound(sp) == 13_162      # single seed: exact


def test_window_and_anchor_ranges():
    """Full RIS geometry: every row holds its local window and the anchor
    prefix on top of the draws; with a 1-key draw the row is exactly their
    union; ppm = 10^6 still gives the causal triangle."""
    for mode in (geo.STOCHASTIC, geo.STRUCTURAL):
        sp = spec(mode=mode, density_ppm=20_000, N=700, n_seeds=3, window=50, anchor=7, block=64)
        row_ptr, col_idx = geo.build_csr(sp)
        check_csr(sp, row_ptr, col_idx)
        for q in range(sp.N):
            row = col_idx[row_ptr[q]:row_ptr[q + 1]]
            assert set(range(max(0, q - 49), q + 1)) <= set(row.tolist())
            assert set(range(0, min(7, q + 1))) <= set(row.tolist())
            assert np.array_equal(row, geo.row_set(sp, 0, q))
    sp = spec(density_ppm=1, N=300, window=20, anchor=5)
    row_ptr, col_idx = geo.build_csr(sp)
    for q in range(sp.N):
        row = set(col_idx[row_ptr[q]:row_ptr[q + 1]].tolist())
        base = set(range(max(0, q - 19), q + 1)) | set(range(0, min(5, q + 1)))
        assert base <= row and len(row - base) <= 1          # one drawn key at most
    sp = spec(density_ppm=10**6, N=200, window=16, anchor=3, n_seeds=2)
    row_ptr, col_idx = geo.build_csr(sp)
    for q in range(sp.N):
        assert np.array_equal(col_idx[row_ptr[q]:row_ptr[q + 1]], np.arange(q + 1))
    sp = spec(density_ppm=30_000, N=900, window=64, anchor=9, n_seeds=4, heads=2)
    assert geo.nnz_upper_bound(sp) >= geo.build_csr(sp)[0][-1]
