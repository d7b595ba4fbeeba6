"""The hot-path step (RoPE from the unrotated inputs, one-pass geometry into a
bound-sized index buffer, sparse attention) recorded into a HIP graph: the
library's calls make no allocation, host synchronisation or memset on that
path, so the step is capturable.  The graph is replayed several times with
eager work and synchronisations between the replays, and every replay must
reproduce the eager step bit for bit."""
import numpy as np
import pytest

from gpu_common import need_gpu, say, torch
from synth import gaussian_qkv, to_bf16

pytestmark = pytest.mark.gpu


def test_hot_path_step_replays_from_a_graph():
    ris = need_gpu()
    Hq, Hkv, N, D, ppm, S = 12, 2, 3000, 128, 20_000, 10
    say(f"graph capture Hq={Hq} Hkv={Hkv} N={N} D={D}")
    Q, K, V = gaussian_qkv(Hq, Hkv, N, D, seed=5)
    q0, k0, v = to_bf16(Q).cuda(), to_bf16(K).cuda(), to_bf16(V).cuda()
    q, k = torch.empty_like(q0), torch.empty_like(k0)
    out = torch.empty(Hq, N, D, dtype=torch.bfloat16, device="cuda")
    rd = ris.rope_desc(ris.ROPE_YARN, 1e6, orig_max_pos=1024)
    md = ris.mask_desc(ris.STOCHASTIC, ppm, N, Hkv, n_seeds=S)
    cap = ris.mask_nnz_bound(md)
    row_ptr = torch.empty(Hkv * N + 1, dtype=torch.int64, device="cuda")
    col_idx = torch.empty(cap, dtype=torch.int32, device="cuda")
    ad = ris.attn_desc(q, k, out)

    def step():
        ris.rope_from(q0, q, rd)
        ris.rope_from(k0, k, rd)
        ris.mask_build(md, row_ptr, col_idx, col_capacity=cap)
        ris.sparse_attn(q, k, v, row_ptr, col_idx, out, ad)

    step()
    torch.cuda.synchronize()
    want_out, want_rp = out.clone(), row_ptr.clone()
    nnz = int(want_rp[-1].item())
    want_ci = col_idx[:nnz].clone()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                      # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for r in range(4):
        out.zero_()
        row_ptr.zero_()
        col_idx.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(row_ptr, want_rp), r
        assert torch.equal(col_idx[:nnz], want_ci), r
        assert torch.equal(out, want_out), r
        # eager work between replays
        step()
        torch.cuda.synchronize()
        assert torch.equal(out, want_out), r
