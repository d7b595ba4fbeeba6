"""Reader of tests/golden/csr_digests.txt (the oracle's full-size geometry
digests) and the geometry descriptors they were written for."""
import importlib.util
import os

HERE = os.path.dirname(os.path.abspath(__file__))
DIGESTS = os.path.join(HERE, "golden", "csr_digests.txt")
_GEN = os.path.join(HERE, "golden", "make_csr_digests.py")

_spec = importlib.util.spec_from_file_location("make_csr_digests", _GEN)
generator = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(generator)
GEOMETRIES = generator.GEOMETRIES
BLOCK_ROWS = generator.BLOCK_ROWS


def load_digests(path=DIGESTS):
    """{(workload, layer): {(kv_head, q0, q1): (nnz, sha256_sizes, sha256_keys)}}"""
    out = {}
    with open(path) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, layer, h, q0, q1, nnz, dsz, dkeys = line.split()
            out.setdefault((name, int(layer)), {})[(int(h), int(q0), int(q1))] = (int(nnz), dsz, dkeys)
    return out
