"""GPU geometry (ris_mask_build) vs the oracle: bit-exact index sets."""
import numpy as np
import pytest

from gpu_common import desc_of, gpu_csr, need_gpu, rows_of, say, spec_of, torch
from oracle import geometry as o_geo

pytestmark = pytest.mark.gpu

SMALL = [
    # mode, ppm, N, heads, S, seed, layer, causal, block[, window, anchor]
    (0, 100_000, 512, 1, 1, 0, 0, 1, 0),           # the tiny workload
    (0, 10_000, 4097, 2, 10, 0, 0, 1, 0),          # ragged N, 10 seeds
    (1, 10_000, 4097, 2, 10, 0, 0, 1, 64),         # Structural, B = 64
    (0, 10_000, 2048, 2, 70, 0, 0, 1, 0),          # 70-seed ensemble
    (1, 50_000, 3000, 4, 10, 0, 5, 1, 64),         # TinyLlama-like, layer 5
    (1, 10_000, 5000, 1, 3, 0, 0, 1, 0),           # paper block rule
    (0, 250_000, 777, 3, 4, 2**63 + 5, 0, 0, 0),   # non-causal, large seed
    (0, 10**6, 300, 2, 3, 0, 0, 1, 0),             # 100%: causal triangle
    (1, 10**6, 300, 1, 2, 0, 0, 1, 7),
    (1, 30_000, 400, 1, 5, 0, 0, 1, 1),            # B = 1: clique is q alone
    (1, 30_000, 400, 1, 5, 0, 0, 1, 1000),         # B > N: one block
    (0, 1, 1000, 1, 300, 9, 2, 1, 0),              # k = 1 rows, 300 seeds (batches of 64)
    (0, 500_000, 1, 1, 4, 0, 0, 1, 0),             # N = 1
    (0, 500_000, 2, 1, 4, 0, 0, 1, 0),             # N = 2
    # full geometry: + window, anchor
    (0, 10_000, 4097, 2, 10, 0, 0, 1, 0, 1024, 4),      # L = 1024 with 4 sink tokens
    (1, 10_000, 4097, 2, 10, 0, 0, 1, 64, 1024, 4),     # window spans many blocks
    (1, 50_000, 3000, 2, 3, 0, 1, 1, 64, 33, 100),      # window inside / across a block
    (0, 1, 1500, 1, 2, 0, 0, 1, 0, 1, 1),               # window and anchor of one key
    (0, 30_000, 700, 1, 4, 0, 0, 1, 0, 5000, 0),        # window wider than N
    (0, 30_000, 700, 1, 4, 0, 0, 1, 0, 0, 800),         # anchor wider than N
    (0, 10**6, 300, 1, 2, 0, 0, 1, 0, 17, 3),           # 100% with ranges: the triangle
]


@pytest.mark.parametrize("fused", [False, True], ids=["two_phase", "one_pass"])
@pytest.mark.parametrize("cfg", SMALL)
def test_mask_bit_exact_small(cfg, fused):
    """Both build paths: count + scan + fill (col_idx sized exactly) and the
    one-pass build (col_idx sized from the closed-form bound)."""
    ris = need_gpu()
    sp = spec_of(*cfg)
    say(f"mask parity {cfg} fused={fused}")
    rp, ci = gpu_csr(ris, sp, use_bound=fused)
    want_rp, want_ci = o_geo.build_csr(sp)
    rp = rp.cpu().numpy()
    assert np.array_equal(rp, want_rp)
    assert np.array_equal(ci.cpu().numpy()[: rp[-1]], want_ci)


def test_mask_bound_sized_fill_and_determinism():
    ris = need_gpu()
    sp = spec_of(0, 10_000, 3000, 2, 10)
    rp1, ci1 = gpu_csr(ris, sp, use_bound=True)
    rp2, ci2 = gpu_csr(ris, sp, use_bound=False)
    nnz = int(rp1[-1].item())
    assert torch.equal(rp1, rp2)
    assert torch.equal(ci1[:nnz], ci2[:nnz])
    rp3, ci3 = gpu_csr(ris, sp)
    assert torch.equal(rp2, rp3) and torch.equal(ci2, ci3)


@pytest.mark.parametrize("use_bound", [False, True], ids=["exact", "bound"])
def test_build_csr_on_a_side_stream(use_bound):
    """Both phases on a caller's stream (not torch's current one), with the
    count read back in between: the CSR equals the default-stream one."""
    ris = need_gpu()
    sp = spec_of(0, 20_000, 4000, 2, 10)
    rp0, ci0 = gpu_csr(ris, sp)
    side = torch.cuda.Stream()
    say(f"side stream build_csr use_bound={use_bound}")
    rp, ci = ris.build_csr(desc_of(ris, sp), "cuda", stream=side, use_bound=use_bound)
    side.synchronize()
    nnz = int(rp0[-1].item())
    assert torch.equal(rp, rp0)
    assert torch.equal(ci[:nnz], ci0[:nnz])


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_mask_into_unaligned_buffer(shift):
    """col_idx starting 1-3 elements past a 16-byte boundary: the rows are
    written with scalar stores up to the first aligned position and 16-byte
    stores after it; every element, and nothing around the written range,
    must come out as from an aligned buffer (one pass and two phases)."""
    ris = need_gpu()
    sp = spec_of(0, 200_000, 1500, 2, 6)
    d = desc_of(ris, sp)
    rp, ci = gpu_csr(ris, sp)
    nnz = int(rp[-1].item())
    cap = ris.mask_nnz_bound(d)
    for use_bound in (True, False):
        base = torch.full((cap + 8,), -5, dtype=torch.int32, device="cuda")
        view = base[shift:shift + (cap if use_bound else nnz)]
        rp2 = torch.empty_like(rp)
        if use_bound:
            ris.mask_build(d, rp2, view, col_capacity=cap)
        else:
            ris.mask_build(d, rp2)
            ris.mask_build(d, rp2, view)
        torch.cuda.synchronize()
        assert torch.equal(rp2, rp)
        assert torch.equal(view[:nnz], ci[:nnz])
        assert bool((base[:shift] == -5).all()) and bool((base[shift + nnz:] == -5).all())


def test_mask_capacity_error_writes_nothing():
    ris = need_gpu()
    sp = spec_of(0, 50_000, 2000, 2, 5)
    d = desc_of(ris, sp)
    rp = torch.empty(sp.heads * sp.N + 1, dtype=torch.int64, device="cuda")
    ris.mask_build(d, rp)
    nnz = int(rp[-1].item())
    small = torch.full((nnz - 1,), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(ris.RisError) as e:
        ris.mask_build(d, rp, small)
    assert e.value.status == ris.E_CAPACITY
    torch.cuda.synchronize()
    assert bool((small == -7).all())
    exact = torch.empty(nnz, dtype=torch.int32, device="cuda")
    ris.mask_build(d, rp, exact)
    assert np.array_equal(exact.cpu().numpy(), o_geo.build_csr(sp)[1])


@pytest.mark.parametrize("name", ["qwen2_32k_stochastic", "qwen2_32k_structural",
                                  "qwen2_64k_stochastic_yarn", "tinyllama_64k_structural",
                                  "qwen2_64k_full_geometry"])
def test_mask_full_size(name):
    """Full-size geometry of each workload: every row's size within its
    closed-form bounds, nnz consistent, sampled rows bit-exact."""
    from synth import WORKLOADS
    from gpu_common import sample_rows
    ris = need_gpu()
    w = WORKLOADS[name]
    layer = 21 if w.layers > 1 else 0
    sp = spec_of(w.mode, w.density_ppm, w.N, w.Hkv, w.n_seeds, w.seed, layer, 1, w.block,
                 w.window, w.anchor)
    say(f"full-size mask {name} layer {layer}")
    rp_d, ci_d = gpu_csr(ris, sp, use_bound=True)
    rp = rp_d.cpu().numpy()
    counts = np.diff(rp)
    q = np.tile(np.arange(w.N), w.Hkv)
    n, kk, start = o_geo._pool_and_draws(sp, q)
    lo, hi = kk.copy(), np.minimum(n, w.n_seeds * kk)
    if w.mode == o_geo.STRUCTURAL:
        lo, hi = lo + (q - start + 1), hi + (q - start + 1)
    if w.window or w.anchor:
        win, anc = np.minimum(w.window, q + 1), np.minimum(w.anchor, q + 1)
        lo = np.maximum(lo, np.maximum(win, anc))
        hi = np.minimum(hi + win + anc, q + 1)
    assert rp[0] == 0 and np.all(counts >= lo) and np.all(counts <= hi)
    rows = sample_rows(w.N, w.Hkv, k_each=10)
    got = rows_of(rp, ci_d, [h * w.N + qq for h, qq in rows])
    for (h, qq), g in zip(rows, got):
        want = o_geo.row_sets(sp, h, np.array([qq]))[0]
        assert np.array_equal(g, want), (h, qq)
    say(f"  nnz = {rp[-1]} ({rp[-1] / (w.Hkv * w.N * (w.N + 1) / 2):.4f} of causal pairs)")


@pytest.mark.parametrize("name", ["qwen2_32k_stochastic", "qwen2_64k_stochastic_yarn"])
def test_union_size_matches_its_expectation(name):
    """Statistical pin of the permutation at full size: with each seed's set
    a uniform k-subset of the pool, a key is in the union with probability
    P = 1 - (1 - k/n)^S (Eq. union coverage), so E[nnz] = sum n P over the
    rows; the inclusion indicators of one row are negatively correlated
    (exact-k draws), so sum n P (1 - P) bounds the variance.  The GPU nnz
    must lie within 5 standard deviations."""
    from synth import WORKLOADS
    ris = need_gpu()
    w = WORKLOADS[name]
    sp = spec_of(w.mode, w.density_ppm, w.N, w.Hkv, w.n_seeds, w.seed, 0, 1)
    say(f"union size {name}")
    rp, _ = gpu_csr(ris, sp, use_bound=True)
    nnz = int(rp[-1].item())
    n = np.arange(1, w.N + 1, dtype=np.float64)
    k = o_geo.row_count(w.density_ppm, n.astype(np.int64)).astype(np.float64)
    P = 1.0 - (1.0 - k / n) ** w.n_seeds
    mean = w.Hkv * float((n * P).sum())
    sd = np.sqrt(w.Hkv * float((n * P * (1.0 - P)).sum()))
    assert abs(nnz - mean) < 5 * sd, (nnz, mean, sd)


def _give_up_case(ris, monkeypatch, env, value, must_poison):
    """Build with a give-up forced from the host (env=value), then check the
    reported result: nothing written past col_idx's capacity; if any row is
    poisoned, the total is -1, the binding's check raises, and every row that
    was not poisoned holds exactly the oracle's keys at its offset.  A build
    with the normal bound afterwards is exact."""
    sp = spec_of(0, 10_000, 16384, 2, 3)
    want_rp, want_ci = o_geo.build_csr(sp)
    d = desc_of(ris, sp)
    cap = ris.mask_nnz_bound(d)
    guard = 4096
    R = sp.heads * sp.N
    rp = torch.empty(R + 1, dtype=torch.int64, device="cuda")
    ci = torch.full((cap + guard,), -7, dtype=torch.int32, device="cuda")
    monkeypatch.setenv(env, str(value))
    ris.mask_build(d, rp, ci, col_capacity=cap)
    torch.cuda.synchronize()
    monkeypatch.delenv(env)
    rp_h, ci_h = rp.cpu().numpy(), ci.cpu().numpy()
    assert (ci_h[cap:] == -7).all(), "write past the capacity"
    counts = np.diff(want_rp)
    poisoned = np.flatnonzero(rp_h[1:] < 0)
    say(f"  total {rp_h[-1]}, {len(poisoned)} of {R} rows poisoned")
    if must_poison:
        assert rp_h[-1] == -1 and len(poisoned) > 0
    if rp_h[-1] >= 0:
        # no row had to wait: the build is complete and exact
        assert len(poisoned) == 0
        assert np.array_equal(rp_h, want_rp) and np.array_equal(ci_h[: rp_h[-1]], want_ci)
    else:
        assert len(poisoned) > 0
        with pytest.raises(ris.RisError) as e:
            ris.check_complete(rp)
        assert e.value.status == ris.E_INCOMPLETE
        good = np.flatnonzero(rp_h[1:R] >= 0)          # rows 0 .. R-2 not poisoned
        assert len(good) > 0
        ends = rp_h[1:][good]
        assert np.array_equal(ends, want_rp[1:][good]), "a row that was not poisoned has a wrong offset"
        for i in range(0, len(good), max(1, len(good) // 200)):
            r, e = good[i], ends[i]
            assert np.array_equal(ci_h[e - counts[r]:e], want_ci[want_rp[r]:want_rp[r + 1]]), r
    rp2, ci2 = gpu_csr(ris, sp, use_bound=True)
    assert np.array_equal(rp2.cpu().numpy(), want_rp)
    assert np.array_equal(ci2.cpu().numpy()[: want_rp[-1]], want_ci)
    return rp_h, poisoned


def test_lookback_give_up_is_reported(monkeypatch):
    """The one-pass build's bounded wait, forced to give up from the host
    (RIS_DEBUG_LOOKBACK_SPINS=0: a row that finds a predecessor not ready
    gives up at once, so every kernel exits normally).  Whether any row has
    to wait depends on the timing; the reported result must be right either
    way."""
    ris = need_gpu()
    say("look-back give-up: N=16384 heads=2 S=3, spin limit 0")
    _give_up_case(ris, monkeypatch, "RIS_DEBUG_LOOKBACK_SPINS", 0, must_poison=False)


def test_forced_poison_row_is_reported(monkeypatch):
    """The poison path whatever the timing: RIS_DEBUG_POISON_ROW makes one
    row publish poison in place of its look-back.  That row and the total
    must read -1, and the rest must be as above."""
    ris = need_gpu()
    r = 2 * 16384 // 3
    say(f"forced poison: N=16384 heads=2 S=3, row {r}")
    rp_h, poisoned = _give_up_case(ris, monkeypatch, "RIS_DEBUG_POISON_ROW", r, must_poison=True)
    assert rp_h[r + 1] == -1 and r in poisoned
    assert (rp_h[1:r + 1] >= 0).all(), "a row before the poisoned one was poisoned"
