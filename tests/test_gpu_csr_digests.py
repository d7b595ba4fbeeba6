"""Full-size geometry, every row of every KV head, against the oracle.

tests/golden/csr_digests.txt holds, per workload geometry, KV head and block of
consecutive query rows, the oracle's entry count and sha256 digests of the row
sizes (int64) and of the keys row after row (int32), written by
tests/golden/make_csr_digests.py, which calls only oracle/ (Methods,
"Memory-Bounded Geometry Generation" and "Sampling Modes"; Results, "Ensemble
Coverage Analysis").  The CSR that the one-pass build writes at full size --
the launch the benchmark times -- is hashed the same way here and must match
every block bit for bit.  The two-phase build (count, scan, fill into a
col_idx of exactly nnz entries) is held to the same digests on two of the
geometries."""
import concurrent.futures
import hashlib

import numpy as np
import pytest

from gpu_common import gpu_csr, need_gpu, say, spec_of
from golden_digests import GEOMETRIES, load_digests

pytestmark = pytest.mark.gpu


def gpu_block_digests(rp, ci, N, heads, blocks):
    """(h, q0, q1) -> (nnz, sha256 of sizes, sha256 of keys) of the GPU CSR."""
    def one(b):
        h, q0, q1 = b
        lo, hi = h * N + q0, h * N + q1
        sizes = np.ascontiguousarray(np.diff(rp[lo:hi + 1]).astype("<i8"))
        keys = np.ascontiguousarray(ci[rp[lo]:rp[hi]])
        return b, (int(rp[hi] - rp[lo]), hashlib.sha256(sizes).hexdigest(),
                   hashlib.sha256(keys.view(np.uint8)).hexdigest())
    with concurrent.futures.ThreadPoolExecutor(max_workers=16) as ex:
        return dict(ex.map(one, blocks))


def check_against_digests(name, layer, use_bound):
    import torch
    ris = need_gpu()
    fields = dict(next(g[2] for g in GEOMETRIES if g[0] == name and g[1] == layer))
    want = load_digests()[(name, layer)]
    sp = spec_of(fields["mode"], fields["density_ppm"], fields["N"], fields["heads"],
                 fields["n_seeds"], fields["seed"], layer, 1, fields.get("block", 0),
                 fields.get("window", 0), fields.get("anchor", 0))
    path = "one-pass" if use_bound else "two-phase"
    say(f"full-size CSR digests {name} layer {layer} ({path}): {len(want)} blocks")
    rp_d, ci_d = gpu_csr(ris, sp, use_bound=use_bound)
    rp = rp_d.cpu().numpy()
    assert rp[0] == 0 and rp[-1] >= 0
    ci = ci_d[: int(rp[-1])].cpu().numpy()
    del ci_d, rp_d
    torch.cuda.empty_cache()
    got = gpu_block_digests(rp, ci, sp.N, sp.heads, list(want))
    bad = [b for b, v in want.items() if got[b] != v]
    say(f"  nnz {rp[-1]}, {len(want) - len(bad)} of {len(want)} blocks identical")
    assert not bad, f"blocks differing from the oracle: {bad[:8]}"
    assert int(rp[-1]) == sum(v[0] for v in want.values())


@pytest.mark.parametrize("name,layer", [(g[0], g[1]) for g in GEOMETRIES],
                         ids=[f"{g[0]}-layer{g[1]}" for g in GEOMETRIES])
def test_full_size_csr_matches_oracle_digests(name, layer):
    check_against_digests(name, layer, use_bound=True)


@pytest.mark.parametrize("name,layer", [("qwen2_32k_structural", 0), ("qwen2_64k_stochastic_yarn", 0)],
                         ids=["qwen2_32k_structural-layer0", "qwen2_64k_stochastic_yarn-layer0"])
def test_two_phase_build_matches_oracle_digests(name, layer):
    check_against_digests(name, layer, use_bound=False)
