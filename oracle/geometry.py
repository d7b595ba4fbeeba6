"""RIS attention geometry: per-row key sets and their CSR (oracle; test only).

Follows the paper's Methods section:

* "Memory-Bounded Geometry Generation": each seed's indices are drawn, filtered
  for causality and merged into one master set; the seed is then discarded.
* "Sampling Modes: Stochastic and Structural": Stochastic treats the whole
  (causal) sequence as one uniform pool; Structural cuts the sequence into
  blocks of size ``B = min(0.1 N, B_max)``, connects each block as a clique and
  adds global edges, with the clique's cost deducted from the global budget.
* Results, "Ensemble Coverage Analysis": the ensemble is the *union* of the
  seeds' index sets (coverage ``U = 1 - (1 - d)^S``).
* "Hybrid Anchor and Pre-Fusion Unified Softmax": the sets merge through
  ``unique()`` before K/V extraction -- every index appears once.

Readings taken where the paper is silent (each also listed in the design notes):

1. Density is relative to the causal pool ``n_q = q + 1`` (the paper draws over
   the sequence and then filters for causality, whose expected kept fraction is
   ``d``); with ``causal = 0`` the pool is ``[0, N)``.
2. The count per row and seed is exact:
   ``k(q) = clamp(floor((ppm * n_q + 500000) / 10^6), 1, n_q)`` -- round half up
   of ``d * n_q`` in integers.  The same rule on ``n = N = 65,536`` reproduces
   every ``B_max`` of the sub-1% sweet-spot table (Results, "Sweet-Spot
   Analysis").  ``k >= 1`` keeps every softmax row non-empty.
3. Structural: block ``b = floor(q / B)``; clique ``C(q) = [bB, q]`` (the causal
   filter applied to the block clique); global count
   ``k_g(q) = min(bB, max(0, k(q) - |C(q)|))`` drawn from ``[0, bB)`` (disjoint
   from the clique).  The clique cost is deducted per row, so a row costs
   exactly ``k(q)`` whenever the clique fits in the budget.
4. ``B = 0`` selects the paper's rule ``B = min(floor(N / 10), B_max)`` with
   ``B_max = k`` evaluated on ``n = N``.
5. Seeds are ``seed, seed + 1, ..., seed + S - 1``; the layer index enters the
   hash, so layers get distinct sets.
6. The hash is keyed by the KV head, so all query heads of a GQA group share
   one set.
7. The full RIS geometry (Methods, "Ensemble Stochastic Projection and
   Retrieval Coverage") also holds a dense local sliding window of L tokens
   and a global anchor over the initial tokens.  Reading: both join the same
   union -- window ``[max(0, q - L + 1), q]``, anchor ``[0, min(A, q + 1))`` --
   on top of the ensemble's draws, whose counts are unchanged; the paper does
   not give A (``anchor = 0`` and ``window = 0`` leave them out).  Causal only.
"""

from dataclasses import dataclass

import numpy as np

from . import philox, prp

STOCHASTIC = 0
STRUCTURAL = 1
PPM = 1_000_000


@dataclass(frozen=True)
class MaskSpec:
    """What a geometry depends on (the oracle's own record of the inputs)."""
    mode: int
    density_ppm: int
    seed: int
    n_seeds: int
    layer: int
    N: int
    heads: int          # KV heads
    causal: int = 1
    block: int = 0      # Structural B; 0 = the paper's rule
    window: int = 0     # dense local window L (0 = none)
    anchor: int = 0     # initial-token anchor A (0 = none)


def row_count(ppm, n):
    """k = clamp(round_half_up(ppm * n / 10^6), 1, n) on integer arrays."""
    n = np.asarray(n, dtype=np.int64)
    k = (np.int64(ppm) * n + PPM // 2) // PPM
    return np.minimum(np.maximum(k, 1), n)


def block_size(spec):
    """Structural block size B (explicit, or the paper's min(0.1 N, B_max))."""
    if spec.block > 0:
        return int(spec.block)
    b_max = int(row_count(spec.density_ppm, spec.N))
    return max(1, min(spec.N // 10, b_max))


def _pool_and_draws(spec, q):
    """Per row: (pool size n, draws per seed kk, clique start) for rows q."""
    q = np.asarray(q, dtype=np.int64)
    if spec.mode == STOCHASTIC:
        n = q + 1 if spec.causal else np.full_like(q, spec.N)
        return n, row_count(spec.density_ppm, n), None
    B = block_size(spec)
    start = (q // B) * B
    clique = q - start + 1
    k = row_count(spec.density_ppm, q + 1)
    kg = np.minimum(start, np.maximum(0, k - clique))
    return start, kg, start


def seed_draws(spec, kv_head, q, s):
    """One seed's drawn (non-clique) keys for row q, unsorted, as int64."""
    n, kk, _ = _pool_and_draws(spec, np.array([q]))
    rk = philox.row_round_keys(np.uint64((spec.seed + s) % 2**64), q, kv_head, spec.layer)
    return prp.draw(int(kk[0]), int(n[0]), rk).astype(np.int64)


def fixed_ranges(spec, q):
    """The row's deterministic ranges: Structural clique, local window and
    initial-token anchor (as (lo, hi) half-open intervals)."""
    out = []
    if spec.mode == STRUCTURAL:
        start = int(_pool_and_draws(spec, np.array([q]))[2][0])
        out.append((start, q + 1))
    if spec.window > 0:
        out.append((max(0, q - spec.window + 1), q + 1))
    if spec.anchor > 0:
        out.append((0, min(spec.anchor, q + 1)))
    return out


def row_set(spec, kv_head, q):
    """I(kv_head, q): sorted, unique union of every seed's set for one row.

    Written as the plain definition (one seed at a time, then ``unique``).
    """
    parts = [seed_draws(spec, kv_head, q, s) for s in range(spec.n_seeds)]
    parts += [np.arange(lo, hi, dtype=np.int64) for lo, hi in fixed_ranges(spec, q)]
    return np.unique(np.concatenate(parts)) if parts else np.zeros(0, np.int64)


def row_sets(spec, kv_head, qs):
    """I(kv_head, q) for many rows at once (same values as ``row_set``).

    Vectorised over every (row, seed, draw) triple of the batch; the union is
    one ``unique`` over (row, key) pairs.
    """
    qs = np.asarray(qs, dtype=np.int64)
    n, kk, start = _pool_and_draws(spec, qs)
    S = spec.n_seeds
    seeds = (np.uint64(spec.seed) + np.arange(S, dtype=np.uint64))
    rk = philox.row_round_keys(seeds[None, :], qs[:, None].astype(np.uint64),
                               np.uint64(kv_head), np.uint64(spec.layer))   # (R, S, 8)
    per_row = kk * S
    total = int(per_row.sum())
    ri = np.repeat(np.arange(len(qs)), per_row)
    within = np.arange(total) - np.repeat(np.cumsum(per_row) - per_row, per_row)
    si = within // np.repeat(np.maximum(kk, 1), per_row)
    j = within % np.repeat(np.maximum(kk, 1), per_row)
    keys = prp.permute(j.astype(np.uint64), rk[ri, si], n[ri].astype(np.uint64)).astype(np.int64)
    stride = np.int64(spec.N + 1)
    ranges_r, ranges_v = [ri], [keys]
    for i, q in enumerate(qs):
        for lo, hi in fixed_ranges(spec, int(q)):
            ranges_r.append(np.full(hi - lo, i, dtype=np.int64))
            ranges_v.append(np.arange(lo, hi, dtype=np.int64))
    ri = np.concatenate(ranges_r)
    keys = np.concatenate(ranges_v)
    u = np.unique(ri.astype(np.int64) * stride + keys)
    rows = u // stride
    vals = u % stride
    bounds = np.searchsorted(rows, np.arange(len(qs) + 1))
    return [vals[bounds[i]:bounds[i + 1]] for i in range(len(qs))]


def build_csr(spec, batch=256):
    """Full CSR: row r = kv_head * N + q; row_ptr int64, col_idx int32."""
    counts = np.zeros(spec.heads * spec.N, dtype=np.int64)
    cols = []
    for h in range(spec.heads):
        for q0 in range(0, spec.N, batch):
            qs = np.arange(q0, min(spec.N, q0 + batch))
            sets = row_sets(spec, h, qs)
            for i, s in enumerate(sets):
                counts[h * spec.N + q0 + i] = len(s)
            cols.extend(sets)
    row_ptr = np.zeros(spec.heads * spec.N + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    col_idx = np.concatenate(cols).astype(np.int32) if cols else np.zeros(0, np.int32)
    return row_ptr, col_idx


def nnz_upper_bound(spec):
    """Closed-form upper bound on nnz: each row's union is at most
    min(pool, S * draws) plus its clique, window and anchor, and never more
    than the row's key span."""
    q = np.arange(spec.N, dtype=np.int64)
    n, kk, start = _pool_and_draws(spec, q)
    per = np.minimum(n, spec.n_seeds * kk)
    if spec.mode == STRUCTURAL:
        per = per + (q - start + 1)
    if spec.window > 0 or spec.anchor > 0:
        per = per + np.minimum(spec.window, q + 1) + np.minimum(spec.anchor, q + 1)
        per = np.minimum(per, q + 1)
    return int(per.sum()) * spec.heads
