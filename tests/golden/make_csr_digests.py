"""Write the oracle's full-size geometry digests to csr_digests.txt.

For every large workload geometry below, the oracle builds every row of every
KV head (``oracle.geometry.row_sets``, the plain definition of the seed
ensemble's union: Methods, "Memory-Bounded Geometry Generation" and "Sampling
Modes"; Results, "Ensemble Coverage Analysis") and records, per KV head and
block of consecutive query rows:

* the number of entries of the block,
* sha256 of the block's row sizes as little-endian int64,
* sha256 of the block's keys, row after row, as little-endian int32.

The GPU tests hash the CSR that ``ris_mask_build`` writes the same way and
compare.  Only ``oracle/`` computes anything here; the descriptors are
written out in full below.

Run from the repository root (one worker process per physical core, one BLAS
thread each):

    python tests/golden/make_csr_digests.py --workers 8
"""
import argparse
import hashlib
import multiprocessing as mp
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import geometry as o_geo  # noqa: E402

OUT = os.path.join(HERE, "csr_digests.txt")
BLOCK_ROWS = 4096

# (name, layer, MaskSpec fields): the geometry of each large workload.
GEOMETRIES = [
    ("qwen2_32k_stochastic", 0, dict(mode=0, density_ppm=10_000, seed=0, n_seeds=10, N=32768, heads=2)),
    ("qwen2_32k_structural", 0, dict(mode=1, density_ppm=10_000, seed=0, n_seeds=10, N=32768, heads=2,
                                     block=64)),
    ("qwen2_64k_stochastic_yarn", 0, dict(mode=0, density_ppm=10_000, seed=0, n_seeds=70, N=65536,
                                          heads=2)),
    ("tinyllama_64k_structural", 0, dict(mode=1, density_ppm=50_000, seed=0, n_seeds=10, N=65536,
                                         heads=4, block=64)),
    ("tinyllama_64k_structural", 21, dict(mode=1, density_ppm=50_000, seed=0, n_seeds=10, N=65536,
                                          heads=4, block=64)),
    ("qwen2_64k_full_geometry", 0, dict(mode=0, density_ppm=10_000, seed=0, n_seeds=70, N=65536, heads=2,
                                        window=1024, anchor=4)),
]


def spec_for(layer, fields):
    return o_geo.MaskSpec(layer=layer, **fields)


def block_digest(task):
    """(name, layer, kv_head, q0, q1) -> digests of rows [q0, q1) of that head."""
    from threadpoolctl import threadpool_limits
    name, layer, fields, h, q0, q1 = task
    spec = spec_for(layer, fields)
    with threadpool_limits(1):
        h_cnt, h_col = hashlib.sha256(), hashlib.sha256()
        counts = np.zeros(q1 - q0, dtype="<i8")
        q = q0
        while q < q1:
            # about three million draws per batch keeps a worker near 0.5 GB
            per_row = max(1, spec.n_seeds * int(o_geo.row_count(spec.density_ppm, q + 1)))
            step = int(max(8, min(1024, 3_000_000 // per_row)))
            qs = np.arange(q, min(q1, q + step))
            for i, s in zip(qs, o_geo.row_sets(spec, h, qs)):
                counts[i - q0] = len(s)
                h_col.update(np.ascontiguousarray(s, dtype="<i4").tobytes())
            q = int(qs[-1]) + 1
        h_cnt.update(counts.tobytes())
    return name, layer, h, q0, q1, int(counts.sum()), h_cnt.hexdigest(), h_col.hexdigest()


def tasks(selected):
    out = []
    for name, layer, fields in GEOMETRIES:
        if selected and name not in selected:
            continue
        N, heads = fields["N"], fields["heads"]
        for h in range(heads):
            for q0 in range(0, N, BLOCK_ROWS):
                out.append((name, layer, fields, h, q0, min(N, q0 + BLOCK_ROWS)))
    # the heaviest blocks (late rows) first
    return sorted(out, key=lambda t: -t[4])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workers", type=int, default=8)
    ap.add_argument("--only", nargs="*", default=[],
                    help="workload names to (re)compute; the other entries of the file are kept")
    args = ap.parse_args()
    t0 = time.time()
    res = []
    if args.only and os.path.exists(OUT):
        for line in open(OUT):
            if line.startswith("#") or not line.strip():
                continue
            f = line.split()
            if f[0] not in args.only:
                res.append((f[0], int(f[1]), int(f[2]), int(f[3]), int(f[4]), int(f[5]), f[6], f[7]))
    with mp.get_context("fork").Pool(args.workers) as pool:
        for i, r in enumerate(pool.imap_unordered(block_digest, tasks(args.only), chunksize=1)):
            res.append(r)
            print(f"[{time.time() - t0:7.1f} s] {r[0]} layer {r[1]} head {r[2]} rows {r[3]}..{r[4]}",
                  flush=True)
    res.sort(key=lambda r: ([g[0] for g in GEOMETRIES].index(r[0]), r[1], r[2], r[3]))
    with open(OUT, "w") as f:
        f.write("# Oracle digests of the full-size geometry CSR (oracle.geometry.row_sets).\n")
        f.write("# Written by: python tests/golden/make_csr_digests.py --workers 8 (every geometry; "
                "--only NAME recomputes one)\n")
        f.write("# Per KV head and block of query rows [q0, q1): entries, sha256 of the row sizes\n")
        f.write("# (little-endian int64) and sha256 of the keys row after row (little-endian int32).\n")
        f.write("# workload layer kv_head q0 q1 nnz sha256_sizes sha256_keys\n")
        for r in res:
            f.write(" ".join(str(x) for x in r) + "\n")
    print(f"wrote {OUT} ({len(res)} blocks) in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    main()
