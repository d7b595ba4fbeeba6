"""Shared helpers for the GPU parity tests (HIP path vs CPU oracle)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import geometry as o_geo  # noqa: E402


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_21927_amd import ris
    ris.lib()          # raises if the HIP library is missing: no fallback
    return ris


def say(msg):
    print(msg, flush=True)


def spec_of(mode, ppm, N, heads, S=1, seed=0, layer=0, causal=1, block=0, window=0, anchor=0):
    return o_geo.MaskSpec(mode=mode, density_ppm=ppm, seed=seed, n_seeds=S, layer=layer, N=N,
                          heads=heads, causal=causal, block=block, window=window, anchor=anchor)


def desc_of(ris, spec):
    return ris.mask_desc(spec.mode, spec.density_ppm, spec.N, spec.heads, n_seeds=spec.n_seeds,
                         seed=spec.seed, layer=spec.layer, causal=spec.causal, block=spec.block,
                         window=spec.window, anchor=spec.anchor)


def gpu_csr(ris, spec, use_bound=False):
    return ris.build_csr(desc_of(ris, spec), "cuda", use_bound=use_bound)


def rows_of(row_ptr_np, col_gpu, rows):
    """Fetch selected CSR rows from a device col_idx (without copying it all)."""
    out = []
    for r in rows:
        a, b = int(row_ptr_np[r]), int(row_ptr_np[r + 1])
        out.append(col_gpu[a:b].cpu().numpy().astype(np.int64))
    return out


def sample_rows(N, heads, k_each=12, seed=0):
    """Row ids (kv_head * N + q): the first and last rows of each head plus
    random ones in between."""
    rng = np.random.default_rng(seed)
    qs = np.unique(np.concatenate([np.arange(min(4, N)), np.arange(max(0, N - 4), N),
                                   rng.integers(0, N, size=k_each)]))
    return [(h, int(q)) for h in range(heads) for q in qs]


def bf16_ulp_tol(y):
    """One bf16 unit in the last place of |y| (half-ulp rounding plus margin)."""
    return np.ldexp(1.0, np.frexp(np.abs(y))[1] - 8)
