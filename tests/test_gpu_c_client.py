"""The C ABI used from plain C++ (tests/c_client/ris_client.cpp, built by the
build step into _build/libris_client.so and called in this process): the
caller allocates its own device buffers, builds the geometry in one pass and
runs the sparse attention.  Its CSR must equal the oracle's bit for bit and
its output meet the bf16 bar."""
import ctypes
import os
import tempfile

import numpy as np
import pytest

from gpu_common import need_gpu, say, spec_of
from oracle import attention as o_att
from oracle import geometry as o_geo
from synth import gaussian_qkv, to_bf16

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT = os.path.join(ROOT, "_build", "libris_client.so")


@pytest.mark.parametrize("Hq,Hkv,N,D,ppm,S", [(12, 2, 1500, 128, 20_000, 10), (32, 4, 700, 64, 50_000, 5)])
def test_c_client_matches_the_oracle(Hq, Hkv, N, D, ppm, S):
    need_gpu()
    if not os.path.exists(CLIENT):
        pytest.fail("the ABI client is not built (run the build step)")
    say(f"C client Hq={Hq} Hkv={Hkv} N={N} D={D} ppm={ppm} S={S}")
    Q, K, V = gaussian_qkv(Hq, Hkv, N, D, seed=3)
    Qb, Kb, Vb = to_bf16(Q), to_bf16(K), to_bf16(V)
    with tempfile.TemporaryDirectory() as d:
        for name, t in (("q", Qb), ("k", Kb), ("v", Vb)):
            t.view(dtype=__import__("torch").int16).numpy().tofile(os.path.join(d, f"{name}.bin"))
        lib = ctypes.CDLL(CLIENT)
        lib.ris_client_run.argtypes = [ctypes.c_char_p, ctypes.c_char_p, ctypes.c_int64, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
        lib.ris_client_run.restype = ctypes.c_int
        assert lib.ris_client_run(d.encode(), d.encode(), N, Hq, Hkv, D, ppm, S) == 0
        rp = np.fromfile(os.path.join(d, "row_ptr.bin"), dtype=np.int64)
        ci = np.fromfile(os.path.join(d, "col_idx.bin"), dtype=np.int32)
        out = np.fromfile(os.path.join(d, "out.bin"), dtype=np.float32).reshape(Hq, N, D)
    sp = spec_of(0, ppm, N, Hkv, S, 0, 0, 1)
    want_rp, want_ci = o_geo.build_csr(sp)
    assert np.array_equal(rp, want_rp)
    assert np.array_equal(ci, want_ci)
    want = o_att.sparse_attention(Qb.float().numpy(), Kb.float().numpy(), Vb.float().numpy(), want_rp, want_ci)
    V_max = float(np.abs(Vb.float().numpy()).max())
    assert np.abs(out - want).max() <= 2.0**-9 * V_max + 2e-4
