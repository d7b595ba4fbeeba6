"""End-to-end hot path at the workloads' full sizes (RoPE -> geometry ->
sparse attention, bf16 in / bf16 out, the launch configuration the benchmark
times), checked on sampled rows the oracle computes one by one.

Bar on the sampled outputs, element by element: the kernels form exact bf16
products with float32 sums and round the softmax weights to bf16 before the
PV product (relative 2^-9 per weight, so at most 2^-9 max|V| on the output),
and the output itself is rounded to bf16 (half an ulp: at most 2^-9 |out|):
|got - want| <= 2^-9 max|V| + 2^-9 |want| + 2e-4."""
import numpy as np
import pytest

from gpu_common import desc_of, need_gpu, rows_of, sample_rows, say, spec_of, torch
from oracle import attention as o_att
from oracle import geometry as o_geo
from oracle import rope as o_rope
from synth import ROPE_NONE, WORKLOADS, gaussian_qkv, needle_plan, plant_needles, to_bf16

pytestmark = pytest.mark.gpu


def gpu_pipeline(ris, w, Qb, Kb, Vb, layer):
    qd, kd, vd = Qb.cuda(), Kb.cuda(), Vb.cuda()
    if w.rope != ROPE_NONE:
        rd = ris.rope_desc(w.rope, w.rope_base, orig_max_pos=w.rope_orig, factor=w.rope_factor)
        ris.rope(qd, rd)
        ris.rope(kd, rd)
    if w.needles:
        Qn = plant_needles(qd.float().cpu().numpy(), kd.float().cpu().numpy(), needle_plan(w.N))
        qd = to_bf16(Qn.astype(np.float32)).cuda()
    sp = spec_of(w.mode, w.density_ppm, w.N, w.Hkv, w.n_seeds, w.seed, layer, 1, w.block,
                 w.window, w.anchor)
    rp, ci = ris.build_csr(desc_of(ris, sp), "cuda", use_bound=True)
    out = torch.empty(w.Hq, w.N, w.D, dtype=torch.bfloat16, device="cuda")
    ris.sparse_attn(qd, kd, vd, rp, ci, out,
                    ris.attn_desc(qd, kd, out, mode=w.mode, block=w.block))
    torch.cuda.synchronize()
    return sp, out


@pytest.mark.parametrize("name", ["qwen2_32k_stochastic", "qwen2_32k_structural",
                                  "qwen2_64k_stochastic_yarn", "tinyllama_64k_structural",
                                  "qwen2_64k_full_geometry"])
def test_workload_end_to_end(name):
    ris = need_gpu()
    w = WORKLOADS[name]
    layer = 21 if w.layers > 1 else 0
    say(f"workload {name}: Hq={w.Hq} Hkv={w.Hkv} N={w.N} D={w.D} layer={layer}")
    Q, K, V = gaussian_qkv(w.Hq, w.Hkv, w.N, w.D, seed=0)
    Qb, Kb, Vb = to_bf16(Q), to_bf16(K), to_bf16(V)
    del Q, K, V
    sp, out = gpu_pipeline(ris, w, Qb, Kb, Vb, layer)

    rows = sample_rows(w.N, w.Hq, k_each=28, seed=1)
    qs = np.array(sorted({q for _, q in rows}))
    Kr = Kb.float().numpy()
    Vr = Vb.float().numpy()
    if w.rope != ROPE_NONE:
        s = o_rope.scale_factor(w.rope_factor, w.N, w.rope_orig) if w.rope != o_rope.PLAIN else 1.0
        rot = dict(kind=w.rope, base=w.rope_base, s=s, orig_max_pos=w.rope_orig)
        Kr = to_bf16(o_rope.apply(Kr, **rot).astype(np.float32)).float().numpy()
        if w.needles:
            Qr = to_bf16(o_rope.apply(Qb.float().numpy(), **rot).astype(np.float32)).float().numpy()
            Qr = to_bf16(plant_needles(Qr, Kr, needle_plan(w.N)).astype(np.float32)).float().numpy()
        else:
            Qr = np.zeros((w.Hq, w.N, w.D), dtype=np.float32)
            Qr[:, qs] = to_bf16(o_rope.apply(Qb.float().numpy()[:, qs], positions=qs, **rot)
                                .astype(np.float32)).float().numpy()
    else:
        Qr = Qb.float().numpy()
    G = w.Hq // w.Hkv
    got = out.float().cpu().numpy()
    v_max = float(np.abs(Vr).max())
    worst = worst_ratio = 0.0
    sets = {}
    for h, q in rows:
        if (h // G, q) not in sets:
            sets[(h // G, q)] = o_geo.row_sets(sp, h // G, np.array([q]))[0]
        I = sets[(h // G, q)]
        want = o_att.attend_one(Qr[h, q], Kr[h // G, I], Vr[h // G, I], 1 / np.sqrt(w.D))
        err = np.abs(got[h, q] - want)
        tol = 2.0**-9 * v_max + 2.0**-9 * np.abs(want) + 2e-4
        worst = max(worst, float(err.max()))
        worst_ratio = max(worst_ratio, float((err / tol).max()))
    say(f"  {len(rows)} sampled rows, max err {worst:.3e}, max err / bar {worst_ratio:.3f}")
    assert worst <= 2e-2
    assert worst_ratio <= 1.0


def test_longest_sequence_end_to_end():
    """The longest supported sequence (RIS_MAX_N = 262,144 tokens) on the
    Qwen2-1.5B layer shape, Stochastic 1% with 10 seeds (AUTO attention):
    about 6.9e9 index entries, so CSR offsets exceed 2^32.  Sampled rows
    against the oracle, and row_ptr consistent with the closed-form bounds."""
    from synth import STOCHASTIC, Workload
    ris = need_gpu()
    w = Workload("qwen2_256k_stochastic", 12, 2, 128, 262144, "bf16", STOCHASTIC, 10_000, 10)
    say(f"longest sequence: Hq={w.Hq} Hkv={w.Hkv} N={w.N} D={w.D}")
    Q, K, V = gaussian_qkv(w.Hq, w.Hkv, w.N, w.D, seed=2)
    Qb, Kb, Vb = to_bf16(Q), to_bf16(K), to_bf16(V)
    del Q, K, V
    qd, kd, vd = Qb.cuda(), Kb.cuda(), Vb.cuda()
    sp = spec_of(w.mode, w.density_ppm, w.N, w.Hkv, w.n_seeds, w.seed, 0, 1)
    rp_d, ci_d = ris.build_csr(desc_of(ris, sp), "cuda", use_bound=True)
    out = torch.empty(w.Hq, w.N, w.D, dtype=torch.bfloat16, device="cuda")
    ris.sparse_attn(qd, kd, vd, rp_d, ci_d, out, ris.attn_desc(qd, kd, out))
    torch.cuda.synchronize()
    rp = rp_d.cpu().numpy()
    assert rp[-1] > 2**32
    counts = np.diff(rp)
    q = np.tile(np.arange(w.N), w.Hkv)
    n, kk, _ = o_geo._pool_and_draws(sp, q)
    assert rp[0] == 0 and np.all(counts >= kk) and np.all(counts <= np.minimum(n, w.n_seeds * kk))
    rows = sample_rows(w.N, w.Hq, k_each=4, seed=3)
    Qr, Kr, Vr = Qb.float().numpy(), Kb.float().numpy(), Vb.float().numpy()
    G = w.Hq // w.Hkv
    got = out.float().cpu().numpy()
    v_max = float(np.abs(Vr).max())
    worst = worst_ratio = 0.0
    for h, qq in rows:
        I = o_geo.row_sets(sp, h // G, np.array([qq]))[0]
        g_idx = rows_of(rp, ci_d, [(h // G) * w.N + qq])[0]
        assert np.array_equal(g_idx, I), (h, qq)
        want = o_att.attend_one(Qr[h, qq], Kr[h // G, I], Vr[h // G, I], 1 / np.sqrt(w.D))
        err = np.abs(got[h, qq] - want)
        worst = max(worst, float(err.max()))
        worst_ratio = max(worst_ratio, float((err / (2.0**-9 * v_max + 2.0**-9 * np.abs(want) + 2e-4)).max()))
    say(f"  {len(rows)} sampled rows, max err {worst:.3e}, max err / bar {worst_ratio:.3f}")
    assert worst <= 2e-2
    assert worst_ratio <= 1.0


def test_needle_recall_structural_32k():
    """Quality probe of the Structural workload's planted pairs (p, i): a
    needle inside query i's block clique is always in I(i); outside it, p is
    drawn by at least one of the S seeds with probability
    1 - (1 - k_g(i) / bB(i))^S (each seed's draw is uniform over the pool
    [0, bB); Methods, "Sampling Modes", Structural, and the capture
    probability of "Ensemble Stochastic Projection and Retrieval Coverage").
    The GPU geometry's recall over every planted pair and both KV heads must
    match the mean of those probabilities within 5 standard errors."""
    ris = need_gpu()
    w = WORKLOADS["qwen2_32k_structural"]
    sp = spec_of(w.mode, w.density_ppm, w.N, w.Hkv, w.n_seeds, w.seed, 0, 1, w.block)
    say("needle recall qwen2_32k_structural")
    rp_d, ci_d = ris.build_csr(desc_of(ris, sp), "cuda", use_bound=True)
    rp = rp_d.cpu().numpy()
    ci = ci_d[: int(rp[-1])].cpu().numpy()
    p, i = needle_plan(w.N)
    n, kg, start = o_geo._pool_and_draws(sp, i)
    inside = p >= start
    prob = np.where(n > 0, 1.0 - (1.0 - kg / np.maximum(n, 1)) ** w.n_seeds, 0.0)
    for g in range(w.Hkv):
        rows = g * w.N + i
        lo, hi = rp[rows], rp[rows + 1]
        hit = np.array([ci[a + np.searchsorted(ci[a:b], pp)] == pp if np.searchsorted(ci[a:b], pp) < b - a
                        else False for a, b, pp in zip(lo, hi, p)])
        assert hit[inside].all()
        out = ~inside
        got, want = hit[out].mean(), prob[out].mean()
        se = np.sqrt((prob[out] * (1 - prob[out])).sum()) / out.sum()
        assert abs(got - want) < 5 * se, (g, got, want, se)
