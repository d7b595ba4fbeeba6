"""The stored full-size geometry digests (tests/golden/csr_digests.txt).

They are written by tests/golden/make_csr_digests.py from oracle/ alone.
Checked here on the CPU: the descriptors are the workloads' own, the file
covers every (KV head, row block) of every geometry, each block's entry count
lies within its closed-form bounds, and the first block of each geometry
recomputed now from the oracle hashes to the stored digests."""
import hashlib

import numpy as np
import pytest

from golden_digests import BLOCK_ROWS, GEOMETRIES, load_digests
from oracle import geometry as o_geo
from synth import WORKLOADS


def spec_of(layer, fields):
    return o_geo.MaskSpec(layer=layer, **fields)


@pytest.fixture(scope="module")
def digests():
    return load_digests()


@pytest.mark.parametrize("name,layer", [(g[0], g[1]) for g in GEOMETRIES])
def test_descriptor_is_the_workloads(name, layer):
    fields = next(g[2] for g in GEOMETRIES if g[0] == name and g[1] == layer)
    w = WORKLOADS[name]
    assert (fields["mode"], fields["density_ppm"], fields["seed"], fields["n_seeds"], fields["N"],
            fields["heads"], fields.get("block", 0)) == (w.mode, w.density_ppm, w.seed, w.n_seeds, w.N,
                                                         w.Hkv, w.block)
    assert (fields.get("window", 0), fields.get("anchor", 0)) == (w.window, w.anchor)
    assert 0 <= layer < w.layers


@pytest.mark.parametrize("name,layer", [(g[0], g[1]) for g in GEOMETRIES])
def test_digests_cover_every_row_within_bounds(digests, name, layer):
    fields = next(g[2] for g in GEOMETRIES if g[0] == name and g[1] == layer)
    sp = spec_of(layer, fields)
    blocks = digests[(name, layer)]
    want = {(h, q0, min(sp.N, q0 + BLOCK_ROWS)) for h in range(sp.heads) for q0 in range(0, sp.N, BLOCK_ROWS)}
    assert set(blocks) == want
    q = np.arange(sp.N, dtype=np.int64)
    n, kk, start = o_geo._pool_and_draws(sp, q)
    lo, hi = kk.copy(), np.minimum(n, sp.n_seeds * kk)
    if sp.mode == o_geo.STRUCTURAL:
        lo, hi = lo + (q - start + 1), hi + (q - start + 1)
    if sp.window or sp.anchor:
        win, anc = np.minimum(sp.window, q + 1), np.minimum(sp.anchor, q + 1)
        lo = np.maximum(lo, np.maximum(win, anc))
        hi = np.minimum(hi + win + anc, q + 1)
    for (h, q0, q1), (nnz, _, _) in blocks.items():
        assert lo[q0:q1].sum() <= nnz <= hi[q0:q1].sum(), (h, q0)


@pytest.mark.parametrize("name,layer", [(g[0], g[1]) for g in GEOMETRIES])
def test_first_block_recomputed(digests, name, layer):
    fields = next(g[2] for g in GEOMETRIES if g[0] == name and g[1] == layer)
    sp = spec_of(layer, fields)
    h = sp.heads - 1
    q1 = min(sp.N, BLOCK_ROWS)
    sets = o_geo.row_sets(sp, h, np.arange(q1))
    sizes = np.array([len(s) for s in sets], dtype="<i8")
    keys = np.concatenate(sets).astype("<i4")
    got = (int(sizes.sum()), hashlib.sha256(sizes.tobytes()).hexdigest(),
           hashlib.sha256(keys.tobytes()).hexdigest())
    assert got == digests[(name, layer)][(h, 0, q1)]
