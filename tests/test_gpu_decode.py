"""GPU Hybrid-Anchor decode step (ris_mask_build_rows + ris_decode_attn) vs
the oracle.

Index sets are bit-exact (the anchor rows); outputs meet the bf16 bar
(2e-2) and the tighter bound the arithmetic gives: the score and value
products are exact bf16 products summed in float32, and the softmax weights
enter the PV product rounded to bf16, a relative perturbation of at most
2^-9 per weight, so outputs move by at most 2^-9 max|V| (+ 2e-4 for the
float32 sums).
"""
import numpy as np
import pytest

from gpu_common import desc_of, need_gpu, say, spec_of, torch
from oracle import decode as o_dec
from oracle import geometry as o_geo
from synth import decode_inputs, to_bf16

pytestmark = pytest.mark.gpu


def tight_tol(V_max):
    return 2.0**-9 * V_max + 2e-4


ROW_CASES = [
    # mode, ppm, N, heads, S, block, window, anchor, q_begin, q_count
    (0, 10_000, 4097, 2, 10, 0, 0, 0, 0, 4097),
    (0, 10_000, 4097, 2, 10, 0, 0, 0, 1000, 333),
    (0, 10_000, 4097, 2, 70, 0, 0, 0, 4096, 1),
    (1, 50_000, 3000, 4, 10, 64, 0, 0, 2999, 1),
    (1, 10_000, 3000, 2, 10, 64, 128, 4, 700, 129),
    (0, 30_000, 2000, 1, 4, 0, 64, 3, 0, 1),
    # the longest sequences: pools across 2^17 (17- to 18-bit domains) and
    # the last rows of RIS_MAX_N
    (0, 10_000, 262144, 1, 3, 0, 0, 0, 131000, 100),
    (0, 2_000, 262144, 2, 5, 0, 0, 0, 262080, 64),
    (1, 10_000, 262144, 1, 3, 64, 1024, 4, 262100, 44),
    # one-pass build with one row in flight per workgroup (bitmaps of 73k to
    # 100k keys; the range below crosses 65536, so both walks run)
    (0, 1_000, 80000, 2, 2, 0, 0, 0, 64000, 16000),
    (1, 2_000, 100000, 1, 3, 64, 0, 0, 99000, 1000),
]


@pytest.mark.parametrize("fused", [False, True], ids=["two_phase", "one_pass"])
@pytest.mark.parametrize("case", ROW_CASES)
def test_mask_rows_bit_exact(case, fused):
    """A row range of the geometry equals the same rows of the definition."""
    ris = need_gpu()
    mode, ppm, N, heads, S, block, window, anchor, q0, nq = case
    sp = spec_of(mode, ppm, N, heads, S, 0, 2, 1, block, window, anchor)
    say(f"mask rows {case} fused={fused}")
    d = desc_of(ris, sp)
    rp = torch.empty(heads * nq + 1, dtype=torch.int64, device="cuda")
    if fused:
        cap = ris.mask_rows_nnz_bound(d, q0, nq)
    else:
        ris.mask_build_rows(d, q0, nq, rp)
        cap = int(rp[-1].item())
    ci = torch.empty(max(cap, 1), dtype=torch.int32, device="cuda")
    ris.mask_build_rows(d, q0, nq, rp, ci, col_capacity=cap)
    rp_h = rp.cpu().numpy()
    ci_h = ci.cpu().numpy()
    assert rp_h[0] == 0
    for h in range(heads):
        want = o_geo.row_sets(sp, h, np.arange(q0, q0 + nq))
        for i, w in enumerate(want):
            r = h * nq + i
            assert np.array_equal(ci_h[rp_h[r]:rp_h[r + 1]], w), (h, q0 + i)


def build_anchor_cache(ris, sp, t0s, Hkv):
    """Per-sequence anchors (row t0 of the seed geometry, no window or
    initial range) built into the slices of one batched cache."""
    from dataclasses import replace
    B = len(t0s)
    descs = [desc_of(ris, replace(sp, window=0, anchor=0)) for _ in t0s]
    stride = max(ris.mask_rows_nnz_bound(d, t0, 1) for d, t0 in zip(descs, t0s))
    aptr = torch.zeros(B * (Hkv + 1), dtype=torch.int64, device="cuda")
    aidx = torch.full((max(B * stride, 1),), -1, dtype=torch.int32, device="cuda")
    for b, (d, t0) in enumerate(zip(descs, t0s)):
        ris.mask_build_rows(d, t0, 1, aptr[b * (Hkv + 1):(b + 1) * (Hkv + 1)],
                            aidx[b * stride:(b + 1) * stride], col_capacity=stride)
    return aptr, aidx, stride


def run_decode(Hq, Hkv, D, mode, ppm, S, block, window, sink, t0s, ts, max_len,
               dtype_out="f32", seed=0, check_anchor=True):
    ris = need_gpu()
    B = len(t0s)
    G = Hq // Hkv
    Q, K, V = decode_inputs(B, Hq, Hkv, max_len, D, seed=seed)
    Qb, Kb, Vb = to_bf16(Q), to_bf16(K), to_bf16(V)
    Qf, Kf, Vf = Qb.float().numpy(), Kb.float().numpy(), Vb.float().numpy()
    sp = spec_of(mode, ppm, max_len, Hkv, S, 0, 3, 1, block, window, sink)
    aptr, aidx, stride = build_anchor_cache(ris, sp, t0s, Hkv)
    qd, kd, vd = Qb.cuda(), Kb.cuda(), Vb.cuda()
    out = torch.empty(B, Hq, D, device="cuda",
                      dtype=torch.float32 if dtype_out == "f32" else torch.bfloat16)
    pos = torch.tensor(ts, dtype=torch.int64, device="cuda")
    dd = ris.decode_desc(qd, kd, out, stride, window=window, sink=sink)
    ws = torch.empty(ris.decode_workspace_bytes(dd), dtype=torch.uint8, device="cuda")
    ris.decode_attn(qd, kd, vd, pos, aptr, aidx, out, ws, dd)
    got = out.float().cpu().numpy()

    want = np.zeros((B, Hq, D))
    aptr_h, aidx_h = aptr.cpu().numpy(), aidx.cpu().numpy()
    for b in range(B):
        for g in range(Hkv):
            anc = o_dec.stochastic_anchor(sp, g, t0s[b])
            if check_anchor:
                lo, hi = aptr_h[b * (Hkv + 1) + g], aptr_h[b * (Hkv + 1) + g + 1]
                assert np.array_equal(aidx_h[b * stride + lo:b * stride + hi], anc), (b, g)
            t = ts[b]
            if not 0 <= t < max_len:
                continue
            idx = o_dec.step_set(anc, t, window, sink)
            want[b, g * G:(g + 1) * G] = o_dec.decode_attention(
                Qf[b, g * G:(g + 1) * G], Kf[b, g], Vf[b, g], idx, 1 / np.sqrt(D))
    return got, want, float(np.abs(Vf).max())


DECODE_CASES = [
    # Hq, Hkv, D, mode, ppm, S, block, window, sink, t0s, ts, max_len, out
    (12, 2, 128, 0, 10_000, 10, 0, 1024, 4, [3000], [3000], 3100, "f32"),      # first step
    (12, 2, 128, 0, 10_000, 10, 0, 1024, 4, [3000, 2048, 100], [3050, 2300, 1500], 3100, "f32"),
    (12, 2, 128, 0, 10_000, 70, 0, 64, 0, [2500, 2900], [2600, 2999], 3000, "bf16"),
    (32, 4, 64, 1, 50_000, 10, 64, 256, 16, [1900, 1000], [1999, 1777], 2000, "f32"),
    (8, 1, 64, 0, 30_000, 4, 0, 0, 0, [1200, 700, 5], [1300, 701, 5], 1400, "f32"),   # anchor only
    (6, 6, 128, 0, 20_000, 3, 0, 1, 1, [800], [1900], 2000, "f32"),           # G = 1
    (16, 2, 128, 0, 5_000, 5, 0, 33, 7, [1500, 1500], [1400, 1600], 1700, "f32"),  # t < t0
]


@pytest.mark.parametrize("case", DECODE_CASES)
def test_decode_matches_oracle(case):
    Hq, Hkv, D, mode, ppm, S, block, window, sink, t0s, ts, max_len, dout = case
    say(f"decode parity {case}")
    got, want, vmax = run_decode(Hq, Hkv, D, mode, ppm, S, block, window, sink, t0s, ts,
                                 max_len, dout)
    err = float(np.abs(got - want).max())
    say(f"  max err {err:.3e}")
    assert err <= 2e-2
    if dout == "f32":
        assert err <= tight_tol(vmax)


def test_decode_out_of_range_positions_give_zeros():
    got, want, _ = run_decode(12, 2, 128, 0, 10_000, 10, 0, 128, 4, [500, 500, 500],
                              [-1, 600, 700], 700, "f32")
    assert np.all(got[0] == 0) and np.all(got[2] == 0)
    assert float(np.abs(got[1] - want[1]).max()) <= 2e-2


def test_decode_window_only_without_anchor():
    """anchor_stride = 0: the set is the window and the initial tokens."""
    ris = need_gpu()
    B, Hq, Hkv, D, L = 2, 12, 2, 128, 300
    Q, K, V = decode_inputs(B, Hq, Hkv, L, D, seed=5)
    Qb, Kb, Vb = to_bf16(Q), to_bf16(K), to_bf16(V)
    qd, kd, vd = Qb.cuda(), Kb.cuda(), Vb.cuda()
    out = torch.empty(B, Hq, D, device="cuda")
    pos = torch.tensor([299, 10], dtype=torch.int64, device="cuda")
    aptr = torch.zeros(B * (Hkv + 1), dtype=torch.int64, device="cuda")
    aidx = torch.zeros(1, dtype=torch.int32, device="cuda")
    dd = ris.decode_desc(qd, kd, out, 0, window=64, sink=4)
    ws = torch.empty(ris.decode_workspace_bytes(dd), dtype=torch.uint8, device="cuda")
    ris.decode_attn(qd, kd, vd, pos, aptr, aidx, out, ws, dd)
    got = out.cpu().numpy()
    Qf, Kf, Vf = Qb.float().numpy(), Kb.float().numpy(), Vb.float().numpy()
    for b, t in enumerate([299, 10]):
        idx = o_dec.step_set(np.zeros(0, np.int64), t, 64, 4)
        for g in range(Hkv):
            w = o_dec.decode_attention(Qf[b, 6 * g:6 * g + 6], Kf[b, g], Vf[b, g], idx, D ** -0.5)
            assert float(np.abs(got[b, 6 * g:6 * g + 6] - w).max()) <= tight_tol(5.5)


def test_decode_deterministic_and_workspace_reuse():
    """Two calls with a dirty workspace give identical bits."""
    ris = need_gpu()
    B, Hq, Hkv, D, L = 3, 12, 2, 128, 2000
    Q, K, V = decode_inputs(B, Hq, Hkv, L, D, seed=2)
    qd, kd, vd = to_bf16(Q).cuda(), to_bf16(K).cuda(), to_bf16(V).cuda()
    sp = spec_of(0, 10_000, L, Hkv, 10, 0, 0, 1, 0, 128, 4)
    aptr, aidx, stride = build_anchor_cache(ris, sp, [1500, 1600, 1700], Hkv)
    pos = torch.tensor([1999, 1800, 1700], dtype=torch.int64, device="cuda")
    out1 = torch.empty(B, Hq, D, device="cuda")
    dd = ris.decode_desc(qd, kd, out1, stride, window=128, sink=4)
    ws = torch.full((ris.decode_workspace_bytes(dd),), 0xAB, dtype=torch.uint8, device="cuda")
    ris.decode_attn(qd, kd, vd, pos, aptr, aidx, out1, ws, dd)
    out2 = torch.empty_like(out1)
    ris.decode_attn(qd, kd, vd, pos, aptr, aidx, out2, ws, dd)
    assert torch.equal(out1, out2)
    small = torch.empty(ws.numel() - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(ris.RisError) as e:
        ris.decode_attn(qd, kd, vd, pos, aptr, aidx, out2, small, dd)
    assert e.value.status == ris.E_CAPACITY


def test_decode_full_size_qwen2_64k():
    """The 64k Qwen2 layer with the full geometry (70 seeds at 1%, window
    1024, 4 initial tokens): 4 sequences whose first generated token sat at
    65,536 - 64, decoding 1..200 tokens later."""
    t0s = [65472, 65472, 65500, 65400]
    ts = [65472, 65500, 65535, 65599]
    got, want, vmax = run_decode(12, 2, 128, 0, 10_000, 70, 0, 1024, 4, t0s, ts, 65600, "bf16")
    err = float(np.abs(got - want).max())
    say(f"  full-size decode max err {err:.3e}")
    assert err <= 2e-2


def test_decode_large_batch_many_tiles_per_wave():
    """64 sequences x 2 kv heads: few waves per row, so every wave walks
    several 32-key tiles (the round-robin split and the prefetch chain)."""
    B = 64
    t0s = [3000 + 13 * b for b in range(B)]
    ts = [t0 + (b % 5) * 40 for b, t0 in enumerate(t0s)]
    got, want, vmax = run_decode(12, 2, 128, 0, 10_000, 10, 0, 1024, 4, t0s, ts, 4100, "f32",
                                 check_anchor=False)
    err = float(np.abs(got - want).max())
    say(f"  batch-64 decode max err {err:.3e}")
    assert err <= tight_tol(vmax)
