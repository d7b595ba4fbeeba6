"""Benchmark of the RIS sparse-attention hot path on one MI355X.

One step = one layer (or, with --all-layers, every layer of the workload back
to back, each with its own geometry) of the hot path over resident synthetic
inputs: RoPE of the unrotated Q and K into the rotated buffers, geometry (the
CSR of the seed-ensemble union, built in one pass into a col_idx sized from
the closed-form bound), sparse attention.  The default workload is the
Qwen2-1.5B-shaped layer at N = 65,536 tokens, 1% density, 70 seeds, YaRN x2 --
the configuration the headline metric names; the default line also carries
one sub-object per other configuration ("workloads": the tiny float32 case,
the 32k Qwen2 layers, the TinyLlama layer over 22 layers, and the Structural
workloads under the paper's own block rule).

Prints ONE JSON line.  `value` is attended (query-head, key) pairs per second
of whole step time; `roofline` is the attention kernel's (the dominant one):
method flops per launch over its HIP-event time against the bf16 MFMA peak.
"""
import argparse
import json
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from synth import (ROPE_LINEAR, ROPE_NONE, ROPE_YARN, STRUCTURAL, WORKLOADS, gaussian_qkv,  # noqa: E402
                   needle_plan, plant_needles)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFS = 2500.0          # dense bf16 matrix peak of MI355X
PROFILES = os.path.join(ROOT, "profiles")
KV_PAIR_BYTES = {128: 2 * 128 * 2 + 4, 64: 2 * 64 * 2 + 4}   # K row + V row (bf16) + int32 index


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, on a bounded row sample.
# ---------------------------------------------------------------------------
_CPU = {}


def _cpu_init(state):
    # One BLAS thread per worker process: oversubscribed BLAS threads saturate
    # the memory bus (the paper's thread-count lesson).
    from threadpoolctl import threadpool_limits
    _CPU["limits"] = threadpool_limits(1)
    _CPU.update(state)


def _cpu_rows(task):
    from oracle import attention as o_att
    from oracle import geometry as o_geo
    s = _CPU
    sp, G, D = s["spec"], s["G"], s["D"]
    g, qs = task
    t0 = time.perf_counter()
    sets = o_geo.row_sets(sp, g, np.asarray(qs))
    pairs = 0
    for q, I in zip(qs, sets):
        Ksel, Vsel = s["Kr"][g, I], s["V"][g, I]      # one gather serves the G heads
        for hh in range(G):
            o_att.attend_one(s["Qr"][g * G + hh, q], Ksel, Vsel, 1 / np.sqrt(D))
            pairs += len(I)
    return pairs, time.perf_counter() - t0


def host_cores():
    """Sockets, physical cores and logical CPUs of the host (lscpu), and the
    physical cores this process may run on (its CPU affinity)."""
    import subprocess
    allowed = os.sched_getaffinity(0)
    try:
        out = subprocess.run(["lscpu", "-p=CPU,CORE,SOCKET"], capture_output=True, text=True,
                             timeout=10).stdout
        rows = [tuple(int(x) for x in ln.split(",")[:3]) for ln in out.splitlines()
                if ln and ln[0].isdigit()]
    except (OSError, ValueError, subprocess.SubprocessError):
        rows = []
    if not rows:
        n = os.cpu_count() or 1
        return {"sockets": None, "physical_cores": None, "logical_cpus": n,
                "physical_cores_available": len(allowed)}
    return {"sockets": len({sk for _, _, sk in rows}), "physical_cores": len({(sk, c) for _, c, sk in rows}),
            "logical_cpus": len(rows),
            "physical_cores_available": len({(sk, c) for cpu, c, sk in rows if cpu in allowed})}


def cpu_baseline(w, layer, Q, K, V, workers, stride, host):
    """Oracle pairs/s over every `stride`-th query row of each KV head."""
    from oracle import geometry as o_geo
    from oracle import rope as o_rope
    t_rope = 0.0
    qs = np.arange(stride - 1, w.N, stride)
    Qr, Kr = Q, K
    if w.rope != ROPE_NONE:
        s = o_rope.scale_factor(w.rope_factor, w.N, w.rope_orig) if w.rope != o_rope.PLAIN else 1.0
        t0 = time.perf_counter()
        Kr = o_rope.apply(K, w.rope, w.rope_base, 0, s, w.rope_orig)
        Qr = np.zeros_like(Q)
        Qr[:, qs] = o_rope.apply(Q[:, qs], w.rope, w.rope_base, 0, s, w.rope_orig, positions=qs)
        # K is rotated once for all rows; charge the sample its share of it.
        t_rope = (time.perf_counter() - t0) * (len(qs) / w.N)
    if w.needles and stride == 1:
        # the same planted inputs as the GPU run (input synthesis, not timed)
        Qr = plant_needles(Qr, Kr, needle_plan(w.N)).astype(np.float32)
    spec = o_geo.MaskSpec(mode=w.mode, density_ppm=w.density_ppm, seed=w.seed,
                          n_seeds=w.n_seeds, layer=layer, N=w.N, heads=w.Hkv, block=w.block,
                          window=w.window, anchor=w.anchor)
    state = dict(spec=spec, G=w.Hq // w.Hkv, D=w.D, Qr=Qr, Kr=Kr, V=V)
    # Heavy rows (large q) first, interleaved over tasks of 8 rows.
    tasks = [(g, list(qs[::-1][i:i + 8])) for g in range(w.Hkv) for i in range(0, len(qs), 8)]
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(workers, initializer=_cpu_init, initargs=(state,)) as pool:
        res = pool.map(_cpu_rows, tasks, chunksize=1)
    wall = time.perf_counter() - t0 + t_rope
    pairs = sum(r[0] for r in res)
    return {"value": pairs / wall, "unit": "pairs/s", "cores": workers, "kind": "oracle",
            "sample": (f"every query row of each KV head ({len(qs) * w.Hkv} rows, " if stride == 1 else
                       f"every {stride}th query row of each KV head ({len(qs) * w.Hkv} rows, ") + (
                      f"{pairs} attended pairs), geometry + RoPE share + attention, "
                      f"{wall:.1f} s wall on {workers} worker processes (one per physical core, "
                      f"one BLAS thread each)"),
            "host": {**host, "workers": workers}}


# ---------------------------------------------------------------------------
# GPU
# ---------------------------------------------------------------------------
def stream_copy_gbs(torch, nbytes=1 << 30, reps=10):
    """Measured device-to-device copy bandwidth (bytes read + written per
    second, GB/s) of a 1 GiB buffer: the practical HBM ceiling."""
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2 * nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b
    return gbs


def run_gpu(w, layers, steps, warmup, algo, seed=0):
    """Time the hot-path step of workload w on the GPU.

    A step = for each layer of `layers`: RoPE of the unrotated Q and K into the
    rotated buffers (the inputs stay as they are, so every step starts from the
    same data), the one-pass geometry into a col_idx sized from the
    closed-form bound, and the sparse attention.  The Structural 32k workload
    plants its needles on the rotated vectors (where the +3 sigma logit gain is
    exact) once, before the timed loop; its step's RoPE pass rotates the
    unrotated inputs into buffers of the same shape, and geometry and attention
    run on the planted ones.  Inputs are resident in HBM; per-phase times come
    from HIP events on the stream the library launches on."""
    import torch
    from paper_2607_21927_amd import ris
    from synth import to_bf16
    dev = torch.device("cuda:0")
    Q, K, V = gaussian_qkv(w.Hq, w.Hkv, w.N, w.D, seed=seed)
    if w.dtype == "bf16":
        q0, k0, v = (to_bf16(x).to(dev) for x in (Q, K, V))
    else:
        q0, k0, v = (torch.from_numpy(x).to(dev) for x in (Q, K, V))
    del Q, K, V
    rd = (ris.rope_desc(w.rope, w.rope_base, orig_max_pos=w.rope_orig, factor=w.rope_factor)
          if w.rope != ROPE_NONE else None)
    q_rot = k_rot = None
    if rd is not None:
        q_rot, k_rot = torch.empty_like(q0), torch.empty_like(k0)
    q_att, k_att = (q_rot, k_rot) if rd is not None else (q0, k0)
    if w.needles:
        ris.rope_from(q0, q_rot, rd)
        ris.rope_from(k0, k_rot, rd)
        planted = plant_needles(q_rot.float().cpu().numpy(), k_rot.float().cpu().numpy(), needle_plan(w.N))
        q_att, k_att = to_bf16(planted.astype(np.float32)).to(dev), k_rot.clone()
        del planted
    out = torch.empty(w.Hq, w.N, w.D, dtype=q0.dtype, device=dev)
    descs = [ris.mask_desc(w.mode, w.density_ppm, w.N, w.Hkv, n_seeds=w.n_seeds, seed=w.seed,
                           layer=layer, block=w.block, window=w.window, anchor=w.anchor)
             for layer in layers]
    # The bound does not depend on the layer index: one buffer serves every layer.
    cap = ris.mask_nnz_bound(descs[0])
    row_ptr = torch.empty(w.Hkv * w.N + 1, dtype=torch.int64, device=dev)
    col_idx = torch.empty(cap, dtype=torch.int32, device=dev)
    ad = ris.attn_desc(q_att, k_att, out, mode=w.mode, block=w.block, algo=algo)
    nnz = [0] * len(descs)

    def step(stamps):
        for i, desc in enumerate(descs):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)] if stamps is not None else None
            if ev:
                ev[0].record()
            if rd is not None:
                ris.rope_from(q0, q_rot, rd)
                ris.rope_from(k0, k_rot, rd)
            if ev:
                ev[1].record()
            # col_idx sized from the closed-form bound: one call builds the CSR.
            ris.mask_build(desc, row_ptr, col_idx, col_capacity=cap)
            if ev:
                ev[2].record()
            ris.sparse_attn(q_att, k_att, v, row_ptr, col_idx, out, ad)
            if ev:
                ev[3].record()
                stamps.append(ev)
            if stamps is None:
                nnz[i] = ris.check_complete(row_ptr)      # every layer's CSR complete

    for _ in range(max(1, warmup)):
        step(None)
    torch.cuda.synchronize()
    t_rope = t_mask = t_attn = 0.0
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    stamps = []
    start.record()
    for _ in range(steps):
        step(stamps)
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    for e0, e1, e2, e3 in stamps:
        t_rope += e0.elapsed_time(e1)
        t_mask += e1.elapsed_time(e2)
        t_attn += e2.elapsed_time(e3)
    if ris.check_complete(row_ptr) != nnz[-1]:
        raise SystemExit("the geometry changed between steps")
    del q0, k0, v, q_rot, k_rot, q_att, k_att, out, row_ptr, col_idx
    torch.cuda.empty_cache()
    return dict(ms_step=total_ms / steps, ms_rope=t_rope / steps, ms_mask=t_mask / steps,
                ms_attn=t_attn / steps, nnz=sum(nnz), layers=len(descs), steps=steps)


def attn_kernel_name(w, algo):
    G = w.Hq // w.Hkv
    if w.dtype != "bf16":
        return f"k_attn_gather<{w.D}>"
    # the tiled kernel's key-block size: 96 keys at D = 128, 128 at D = 64
    return f"k_attn_gather16<{w.D}>" if algo == 1 else f"k_attn_tile16<{w.D}, {G}, {96 if w.D == 128 else 128}>"


def attn_roofline(w, g, algo, traffic=None):
    """Roofline of one attention launch (one layer), from the HIP-event time
    of ris_sparse_attn averaged over the timed launches.

    The tiled kernel (bf16, every tile above the dispatch threshold) runs the
    score and PV contractions on MFMA and reads each 64-key K/V block once per
    32 rows x G heads from LDS, so its bound is the matrix unit: `achieved` =
    the method's flops (4 D per attended (query head, key) pair: QK^T and PV)
    per second against the dense bf16 peak.  `issued_dense_frac` prices the
    masked-dense work it issues over every touched block (all causal pairs);
    `traffic` and `hbm_traffic_frac` are the HBM bytes per launch from the
    committed rocprofv3 counters of this kernel source (null when none match);
    `effective_kv_gbs` is the K/V bytes the method reads per second (2 D x 2 B
    + 4 B per kv-pair), an effective rate, not an HBM one.
    The float32 gather kernel is priced against HBM."""
    G = w.Hq // w.Hkv
    t = g["ms_attn"] / g["layers"] * 1e-3
    kv = g["nnz"] / g["layers"]
    if w.dtype == "bf16" and algo != 1:
        flops = kv * G * 4 * w.D
        dense = w.Hq * w.N * (w.N + 1) / 2 * 4 * w.D
        return {"bound": "mfma", "kernel": attn_kernel_name(w, algo),
                "achieved": flops / t / 1e12, "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                "frac": flops / t / 1e12 / MFMA_BF16_PEAK_TFS, "traffic": traffic,
                "flops_per_launch": flops, "issued_dense_flops_per_launch": dense,
                "issued_dense_frac": dense / t / 1e12 / MFMA_BF16_PEAK_TFS,
                "hbm_traffic_gbs": traffic / t / 1e9 if traffic else None,
                "hbm_traffic_frac": traffic / t / 1e9 / HBM_PEAK_GBS if traffic else None,
                "effective_kv_gbs": kv * KV_PAIR_BYTES[w.D] / t / 1e9}
    per_pair = 2 * w.D * (2 if w.dtype == "bf16" else 4) + 4
    achieved = kv * per_pair / t / 1e9
    return {"bound": "hbm", "kernel": attn_kernel_name(w, algo), "achieved": achieved,
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
            "bytes_per_kv_pair": per_pair}


def workload_record(w, g, algo, extra=None):
    """Per-workload figures of one timed run (a sub-object of the JSON line)."""
    G = w.Hq // w.Hkv
    pairs = g["nnz"] * G
    rec = {"workload": w.name, "Hq": w.Hq, "Hkv": w.Hkv, "head_dim": w.D, "N": w.N, "dtype": w.dtype,
           "mode": "structural" if w.mode == STRUCTURAL else "stochastic",
           "density": w.density_ppm / 1e6, "seeds": w.n_seeds, "block": w.block,
           "rope": ["none", "plain", "linear", "yarn"][w.rope + 1], "needles": w.needles,
           "layers": g["layers"], "steps": g["steps"],
           "ms_step": g["ms_step"], "ms_attn": g["ms_attn"], "ms_geometry": g["ms_mask"], "ms_rope": g["ms_rope"],
           "ms_attn_per_layer": g["ms_attn"] / g["layers"],
           "pairs_per_s": pairs / (g["ms_step"] * 1e-3), "attn_pairs_per_s": pairs / (g["ms_attn"] * 1e-3),
           "kv_pairs": g["nnz"], "union_fraction": g["nnz"] / (g["layers"] * w.Hkv * w.N * (w.N + 1) / 2),
           "roofline": attn_roofline(w, g, algo)}
    if extra:
        rec.update(extra)
    return rec


def kv_gather_figure(w, reps=5):
    """The gather kernel on the workload's own shape and density with a single
    seed (the union then stays below the tiled kernel's threshold, so every
    row takes the per-row K/V gather).  `effective_gbs` is algorithmic K/V
    bytes per second; `llc_hbm_gbs` the bytes the committed counters of this
    kernel source put past the L2 caches per second (served by the 256 MB
    last-level cache and HBM together: per-head K/V of 33.6 MB fits the
    last-level cache, and the counters do not split the two)."""
    import torch
    from paper_2607_21927_amd import ris
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(1)
    q = torch.randn(w.Hq, w.N, w.D, generator=gen, device=dev).to(torch.bfloat16)
    k = torch.randn(w.Hkv, w.N, w.D, generator=gen, device=dev).to(torch.bfloat16)
    v = torch.randn(w.Hkv, w.N, w.D, generator=gen, device=dev).to(torch.bfloat16)
    d = ris.mask_desc(w.mode, w.density_ppm, w.N, w.Hkv, n_seeds=1, seed=w.seed, block=w.block)
    rp, ci = ris.build_csr(d, dev, use_bound=True)
    nnz = int(rp[-1].item())
    out = torch.empty_like(q)
    ad = ris.attn_desc(q, k, out, mode=w.mode, block=w.block, algo=ris.ATTN_GATHER)
    for _ in range(2):
        ris.sparse_attn(q, k, v, rp, ci, out, ad)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        ris.sparse_attn(q, k, v, rp, ci, out, ad)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del q, k, v, rp, ci, out
    torch.cuda.empty_cache()
    effective = nnz * KV_PAIR_BYTES[w.D] / (ms * 1e-3) / 1e9
    past_l2 = measured_traffic(f"attn_gather16_{w.name}_1seed", "paper_2607_21927_amd/csrc/attn_gather.hip")
    return {"kernel": f"k_attn_gather16<{w.D}>", "seeds": 1,
            "union_fraction": nnz / (w.Hkv * w.N * (w.N + 1) / 2), "kv_pairs": nnz, "ms": ms,
            "effective_gbs": effective, "bytes_per_kv_pair": KV_PAIR_BYTES[w.D],
            "llc_hbm_bytes_per_launch": past_l2,
            "llc_hbm_gbs": past_l2 / (ms * 1e-3) / 1e9 if past_l2 else None,
            "llc_hbm_frac_of_hbm_peak": past_l2 / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS if past_l2 else None}


def measured_traffic(record, kernel_source):
    """Bytes per launch past the L2 caches (FETCH_SIZE + WRITE_SIZE, each
    scaled by its reading for a device copy of known size) from the committed
    rocprofv3 counter record profiles/<record>_traffic.txt, or None when no
    record exists or the kernel source or the device headers it includes
    changed since the counters were taken."""
    import hashlib
    path = os.path.join(PROFILES, f"{record}_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = dict(line.strip().split("=", 1) for line in open(path)
               if "=" in line and not line.startswith("#"))
    src = os.path.join(ROOT, rec.get("source", ""))
    if not os.path.exists(src) or rec.get("source") != kernel_source:
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec.get("source_sha256"):
        return None
    # the device headers the kernel includes (inline helpers such as the
    # dispatch decision live there), hashed one after the other
    heads = [h for h in rec.get("headers", "").split(",") if h]
    if not heads:
        return None
    hh = hashlib.sha256()
    for h in heads:
        hp = os.path.join(ROOT, h)
        if not os.path.exists(hp):
            return None
        hh.update(open(hp, "rb").read())
    if hh.hexdigest() != rec.get("headers_sha256"):
        return None
    return float(rec["traffic_bytes"])


# ---------------------------------------------------------------------------
# Decode step (Hybrid Anchor): --decode
# ---------------------------------------------------------------------------
def decode_pairs(aptr, aidx, stride, t0s, ts, Hkv, window, sink):
    """kv-pairs attended by one decode step: per (sequence, kv head) the
    anchor entries outside the window and the initial range, plus both."""
    total = 0
    for b, t in enumerate(ts):
        w_lo = max(0, t - window + 1) if window > 0 else t + 1
        s_hi = min(sink, w_lo)
        for g in range(Hkv):
            lo, hi = aptr[b * (Hkv + 1) + g], aptr[b * (Hkv + 1) + g + 1]
            a = aidx[b * stride + lo:b * stride + hi]
            total += int(((a >= s_hi) & (a < w_lo)).sum()) + (t + 1 - w_lo) + s_hi
    return total


def cpu_decode_baseline(w, t0s, ts, Q, K, V, rows):
    """The oracle's decode step on a few (sequence, kv head) rows."""
    from oracle import decode as o_dec
    from oracle import geometry as o_geo
    sp = o_geo.MaskSpec(mode=w.mode, density_ppm=w.density_ppm, seed=w.seed,
                        n_seeds=w.n_seeds, layer=0, N=K.shape[2], heads=w.Hkv, block=w.block)
    G = w.Hq // w.Hkv
    t0 = time.perf_counter()
    pairs = 0
    for b, g in rows:
        anc = o_dec.stochastic_anchor(sp, g, t0s[b])
        idx = o_dec.step_set(anc, ts[b], w.window, w.anchor)
        o_dec.decode_attention(Q[b, g * G:(g + 1) * G], K[b, g], V[b, g], idx, w.D ** -0.5)
        pairs += len(idx) * G
    wall = time.perf_counter() - t0
    return {"value": pairs / wall, "unit": "pairs/s", "cores": 1, "kind": "oracle",
            "sample": f"{len(rows)} (sequence, kv head) rows of the decode step: anchor "
                      f"geometry + merge + attention, {wall:.1f} s on one core"}


def run_decode_bench(w, B, steps, warmup, cpu):
    import torch
    from paper_2607_21927_amd import ris
    dev = torch.device("cuda:0")
    G = w.Hq // w.Hkv
    N = w.N
    max_len = N + steps + warmup + 1
    # Prompts of different lengths: sequence b generated its first token at
    # N - 97 b, so the anchors differ between sequences.
    t0s = [N - 97 * b for b in range(B)]
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    Q = torch.randn(B, w.Hq, w.D, generator=gen, device=dev).to(torch.bfloat16)
    K = torch.randn(B, w.Hkv, max_len, w.D, generator=gen, device=dev).to(torch.bfloat16)
    V = torch.randn(B, w.Hkv, max_len, w.D, generator=gen, device=dev).to(torch.bfloat16)
    md = ris.mask_desc(w.mode, w.density_ppm, max_len, w.Hkv, n_seeds=w.n_seeds, seed=w.seed,
                       layer=0, block=w.block)
    stride = max(ris.mask_rows_nnz_bound(md, t0, 1) for t0 in t0s)
    aptr = torch.zeros(B * (w.Hkv + 1), dtype=torch.int64, device=dev)
    aidx = torch.zeros(B * stride, dtype=torch.int32, device=dev)
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record()
    for b, t0 in enumerate(t0s):
        ris.mask_build_rows(md, t0, 1, aptr[b * (w.Hkv + 1):(b + 1) * (w.Hkv + 1)],
                            aidx[b * stride:(b + 1) * stride], col_capacity=stride)
    a1.record()
    out = torch.empty(B, w.Hq, w.D, dtype=torch.bfloat16, device=dev)
    dd = ris.decode_desc(Q, K, out, stride, window=w.window, sink=w.anchor)
    ws = torch.empty(ris.decode_workspace_bytes(dd), dtype=torch.uint8, device=dev)
    aptr_h, aidx_h = aptr.cpu().numpy(), aidx.cpu().numpy()
    # Each step decodes the next token: position t0 + step.
    positions = [torch.tensor([t0 + i for t0 in t0s], dtype=torch.int64, device=dev)
                 for i in range(warmup + steps)]
    pairs = sum(decode_pairs(aptr_h, aidx_h, stride, t0s, [t0 + warmup + i for t0 in t0s],
                             w.Hkv, w.window, w.anchor) for i in range(steps))
    for i in range(warmup):
        ris.decode_attn(Q, K, V, positions[i], aptr, aidx, out, ws, dd)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        ris.decode_attn(Q, K, V, positions[warmup + i], aptr, aidx, out, ws, dd)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    kv_pairs = pairs / steps
    achieved = kv_pairs * KV_PAIR_BYTES[w.D] / (ms * 1e-3) / 1e9
    if cpu:
        rows = [(0, 0), (B - 1, w.Hkv - 1)]
        Kh = K[[b for b, _ in rows]].float().cpu().numpy()
        cpu_res = cpu_decode_baseline(
            w, [t0s[b] for b, _ in rows], [t0s[b] + warmup for b, _ in rows],
            Q[[b for b, _ in rows]].float().cpu().numpy(), Kh,
            V[[b for b, _ in rows]].float().cpu().numpy(), [(i, g) for i, (_, g) in enumerate(rows)])
    else:
        cpu_res = None
    return {
        "metric": "decode attended (q,k) pairs/s (Hybrid-Anchor step, batch of sequences)",
        "value": kv_pairs * G / (ms * 1e-3),
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: Gaussian Q and K/V caches (torch.randn, seed 0)",
        "config": {"workload": w.name + "_decode", "batch": B, "Hq": w.Hq, "Hkv": w.Hkv,
                   "head_dim": w.D, "first_token_positions": f"{t0s[-1]}..{t0s[0]}",
                   "density": w.density_ppm / 1e6, "seeds": w.n_seeds, "window": w.window,
                   "sink": w.anchor},
        "tokens_per_s": B / (ms * 1e-3),
        "kv_pairs_per_step": kv_pairs,
        "ms_anchor_build_once": a0.elapsed_time(a1),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "k_decode_partial", "bytes_per_kv_pair": KV_PAIR_BYTES[w.D]},
        "cpu_baseline": cpu_res,
    }


# ---------------------------------------------------------------------------
# Model-level prefill (random weights): --model
# ---------------------------------------------------------------------------
class PhaseTimer:
    """HIP events between phase marks; time from one mark to the next is
    charged to the later mark's name."""

    def __init__(self, torch):
        self.torch = torch
        self.marks = []

    def mark(self, name):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record()
        self.marks.append((name, e))

    def totals(self):
        self.torch.cuda.synchronize()
        out = {}
        for (_, a), (name, b) in zip(self.marks, self.marks[1:]):
            out[name] = out.get(name, 0.0) + a.elapsed_time(b)
        return out


MODEL_WORKLOAD = {"qwen2_1.5b": "qwen2_64k_stochastic_yarn", "tinyllama_1.1b": "tinyllama_64k_structural"}


def run_model_bench(name, layers, steps, warmup):
    import torch
    from paper_2607_21927_amd import ris
    from paper_2607_21927_amd.model import PrefillModel
    from synth import MODELS
    cfg = MODELS[name] if not layers else MODELS[name].with_layers(layers)
    w = WORKLOADS[MODEL_WORKLOAD[name]]
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)

    def rnd(*shape, std=0.02, mean=0.0):
        return (torch.randn(*shape, generator=gen, device=dev) * std + mean).to(torch.bfloat16)

    qd, kd = cfg.heads * cfg.head_dim, cfg.kv_heads * cfg.head_dim
    W = {"embed": rnd(cfg.vocab, cfg.hidden), "layers": [], "norm": rnd(cfg.hidden, std=0.1, mean=1.0)}
    for _ in range(cfg.layers):
        L = {"q": rnd(qd, cfg.hidden), "k": rnd(kd, cfg.hidden), "v": rnd(kd, cfg.hidden),
             "o": rnd(cfg.hidden, qd), "gate": rnd(cfg.inter, cfg.hidden), "up": rnd(cfg.inter, cfg.hidden),
             "down": rnd(cfg.hidden, cfg.inter), "ln1": rnd(cfg.hidden, std=0.1, mean=1.0),
             "ln2": rnd(cfg.hidden, std=0.1, mean=1.0)}
        if cfg.qkv_bias:
            L.update(bq=rnd(qd), bk=rnd(kd), bv=rnd(kd))
        W["layers"].append(L)
    model = PrefillModel(cfg, W, dev, torch.bfloat16)
    del W
    N = w.N
    ids = torch.randint(0, cfg.vocab, (N,), generator=gen, device=dev)
    mask = dict(mode=w.mode, density_ppm=w.density_ppm, n_seeds=w.n_seeds, block=w.block)
    runs = {}
    for kind, label in [(ROPE_YARN, "yarn"), (ROPE_LINEAR, "linear")]:
        rd = ris.rope_desc(kind, cfg.rope_base, orig_max_pos=cfg.native_len)
        for _ in range(warmup):
            model.prefill(ids, mask, rd)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            out = model.prefill(ids, mask, rd)
        e1.record()
        torch.cuda.synchronize()
        runs[label] = {"ms": e0.elapsed_time(e1) / steps, "out": out.float()}
    timer = PhaseTimer(torch)
    timer.mark("start")
    model.prefill(ids, mask, ris.rope_desc(ROPE_YARN, cfg.rope_base, orig_max_pos=cfg.native_len),
                  timers=timer)
    timer.mark("proj")
    phases = timer.totals()
    a, b = runs["yarn"]["out"], runs["linear"]["out"]
    rel = float((a - b).norm() / a.norm())
    ms = runs["yarn"]["ms"]
    return {
        "metric": "model-level prefill tokens/s (random-weight decoder stack, RIS attention)",
        "value": N / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: random weights and token ids (torch.randn / randint, seed 0)",
        "config": {"workload": f"{name}_prefill_{N}", "layers": cfg.layers, "hidden": cfg.hidden,
                   "geometry": MODEL_WORKLOAD[name], "rope": "yarn (factor N / native)"},
        "phase_ms_per_prefill": {k: v for k, v in phases.items()},
        "ablation_rope": {"yarn_ms": runs["yarn"]["ms"], "linear_ms": runs["linear"]["ms"],
                          "relative_l2_difference_of_final_states": rel},
        "roofline": None,
        "cpu_baseline": None,
    }


# The configurations timed beside the headline one, one sub-object each in
# the JSON line: the tiny float32 case, the 32k Qwen2 layers (Stochastic, and
# Structural with needles), the TinyLlama layer over all 22 layers, and the
# Structural workloads with the paper's own block rule.
# The oracle's own timing beside each: every row of the tiny and 32k
# workloads, every 64th row (of layer 0) for the 64k ones.
CPU_STRIDE = {"tiny": 1, "qwen2_32k_stochastic": 1, "qwen2_32k_structural": 1,
              "tinyllama_64k_structural": 64, "qwen2_32k_structural_paper_block": 1,
              "tinyllama_64k_structural_paper_block": 64}
OTHER_WORKLOADS = [("tiny", False, 20), ("qwen2_32k_stochastic", False, 10),
                   ("qwen2_32k_structural", False, 10), ("tinyllama_64k_structural", True, 3),
                   ("qwen2_32k_structural_paper_block", False, 10),
                   ("tinyllama_64k_structural_paper_block", False, 5)]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen2_64k_stochastic_yarn", choices=sorted(WORKLOADS))
    ap.add_argument("--layer", type=int, default=0)
    ap.add_argument("--all-layers", action="store_true",
                    help="one step = every layer of the workload back to back (layer 0..L-1)")
    ap.add_argument("--algo", type=int, default=0, help="0 auto, 1 gather, 2 tile")
    ap.add_argument("--cpu-workers", type=int, default=16,
                    help="most oracle worker processes (one per available physical core)")
    ap.add_argument("--cpu-stride", type=int, default=64)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the named workload (no per-configuration sub-objects)")
    ap.add_argument("--decode", action="store_true",
                    help="time the Hybrid-Anchor decode step instead of the prefill layer")
    ap.add_argument("--batch", type=int, default=32, help="sequences per decode step")
    ap.add_argument("--model", choices=sorted(MODEL_WORKLOAD),
                    help="time a model-level prefill of the named random-weight stack")
    ap.add_argument("--model-layers", type=int, default=0, help="layers of the stack (0 = all)")
    ap.add_argument("--kv-gather", action="store_true",
                    help="time only the per-row K/V gather kernel (workload shape, one seed)")
    ap.add_argument("--no-kv-gather", action="store_true",
                    help="leave the K/V gather figure out of the line (profiling runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the hot path needs no cross-GPU exchange and this "
              "build has no multi-GPU launch (run with --gpus 1).", file=sys.stderr)
        sys.exit(2)
    if args.model:
        print(json.dumps(run_model_bench(args.model, args.model_layers, args.steps, args.warmup)))
        return
    if args.kv_gather:
        w = WORKLOADS[args.workload]
        f = kv_gather_figure(w, reps=args.steps)
        import torch
        f["measured_copy_gbs"] = stream_copy_gbs(torch)
        print(json.dumps({"metric": "K/V gather rate (algorithmic K/V bytes / kernel time)",
                          "value": f["effective_gbs"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
                          "warmup": 2, "ms_per_step": f["ms"], "higher_is_better": True,
                          "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
                          "data": "synthetic: Gaussian Q/K/V (torch.randn, seed 1)",
                          "config": {"workload": w.name + "_1seed", "N": w.N, "Hq": w.Hq, "Hkv": w.Hkv,
                                     "head_dim": w.D, "density": w.density_ppm / 1e6, "seeds": 1},
                          "roofline": {"bound": "hbm", "achieved": f["llc_hbm_gbs"], "peak": HBM_PEAK_GBS,
                                       "unit": "GB/s", "frac": f["llc_hbm_frac_of_hbm_peak"],
                                       "traffic": f["llc_hbm_bytes_per_launch"], "kernel": f["kernel"],
                                       "note": "bytes past the L2 caches (last-level cache and HBM)"},
                          "kv_gather": f}))
        return
    if args.decode:
        wl = args.workload if args.workload != "qwen2_64k_stochastic_yarn" else "qwen2_64k_full_geometry"
        print(json.dumps(run_decode_bench(WORKLOADS[wl], args.batch, args.steps, args.warmup,
                                          not args.no_cpu_baseline)))
        return
    w = WORKLOADS[args.workload]

    with_others = not args.headline_only and not args.all_layers and args.workload == "qwen2_64k_stochastic_yarn"
    cpu, cpu_others = None, {}
    if not args.no_cpu_baseline:
        # Before any GPU call: the worker pool forks this process.
        host = host_cores()
        workers = max(1, min(args.cpu_workers, host["physical_cores_available"]))
        todo = [(w, args.cpu_stride)] + ([(WORKLOADS[n], CPU_STRIDE[n]) for n, _, _ in OTHER_WORKLOADS]
                                         if with_others else [])
        for wc, stride in todo:
            from synth import to_bf16
            Q, K, V = gaussian_qkv(wc.Hq, wc.Hkv, wc.N, wc.D, seed=0)
            Qb, Kb, Vb = ((to_bf16(x).float().numpy() for x in (Q, K, V)) if wc.dtype == "bf16"
                          else (Q, K, V))
            del Q, K, V
            c = cpu_baseline(wc, args.layer if wc is w else 0, Qb, Kb, Vb, workers, stride, host)
            del Qb, Kb, Vb
            if wc is w:
                cpu = c
            else:
                cpu_others[wc.name] = c
            print(f"bench: oracle baseline {wc.name} {c['value']:.3e} pairs/s on {workers} workers",
                  file=sys.stderr, flush=True)

    layers = list(range(w.layers)) if args.all_layers else [args.layer]
    g = run_gpu(w, layers, args.steps, args.warmup, args.algo)
    print(f"bench: {w.name} {g['ms_step']:.3f} ms per step", file=sys.stderr, flush=True)
    G = w.Hq // w.Hkv
    pairs = g["nnz"] * G
    tiled = w.dtype == "bf16" and args.algo != 1
    traffic = measured_traffic(f"attn_tile_{w.name}", "paper_2607_21927_amd/csrc/attn_tile.hip") if tiled else None
    gather = (kv_gather_figure(w) if w.dtype == "bf16" and not args.all_layers and not args.no_kv_gather
              else None)
    rec = workload_record(w, g, args.algo)
    import torch
    copy_gbs = stream_copy_gbs(torch)
    roof = attn_roofline(w, g, args.algo, traffic)
    roof["measured_copy_gbs"] = copy_gbs
    res = {
        "metric": "attended (q,k) pairs/s (whole hot-path step: RoPE + geometry + attention)",
        "value": pairs / (g["ms_step"] * 1e-3),
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": g["ms_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic: Gaussian Q/K/V (numpy default_rng(0)) at the layer shape",
        "config": {"workload": w.name, "Hq": w.Hq, "Hkv": w.Hkv, "head_dim": w.D, "N": w.N,
                   "mode": rec["mode"], "density": w.density_ppm / 1e6, "seeds": w.n_seeds, "block": w.block,
                   "window": w.window, "anchor": w.anchor, "rope": rec["rope"],
                   **({"layers": f"0..{len(layers) - 1}"} if len(layers) > 1 else {"layer": args.layer})},
        "ms_per_layer_attn": g["ms_attn"] / len(layers),
        "ms_attn": g["ms_attn"],
        "ms_geometry": g["ms_mask"],
        "ms_rope": g["ms_rope"],
        "attn_pairs_per_s": pairs / (g["ms_attn"] * 1e-3),
        "kv_pairs": g["nnz"],
        "union_fraction": rec["union_fraction"],
        "roofline": roof,
        # The per-row K/V gather path (sparse unions), on this shape with one seed.
        "kv_gather": gather,
        "cpu_baseline": cpu,
    }
    if with_others:
        others = []
        for name, all_layers, steps in OTHER_WORKLOADS:
            wo = WORKLOADS[name]
            lo = list(range(wo.layers)) if all_layers else [0]
            go = run_gpu(wo, lo, steps, 1, 0)
            print(f"bench: {name} {go['ms_step']:.3f} ms per step", file=sys.stderr, flush=True)
            extra = {"block_resolved": block_of(wo)}
            tr = measured_traffic(f"attn_tile_{wo.name}", "paper_2607_21927_amd/csrc/attn_tile.hip")
            if tr:
                t = go["ms_attn"] / go["layers"] * 1e-3
                extra["attn_traffic_per_launch"] = {"bytes": tr, "gbs": tr / t / 1e9,
                                                    "frac_of_hbm_peak": tr / t / 1e9 / HBM_PEAK_GBS,
                                                    "note": "layer 0's counters (profiles/)"}
            if wo.needles:
                extra["needle_note"] = ("needles planted once on the rotated inputs before the timed loop; "
                                        "the step's RoPE pass rotates the unrotated inputs into buffers of "
                                        "the same shape")
            rec_o = workload_record(wo, go, 0, extra)
            rec_o["cpu_baseline"] = cpu_others.get(name)
            others.append(rec_o)
        res["workloads"] = others
    print(json.dumps(res))


def block_of(w):
    """The Structural block size a workload resolves to (the paper's rule when
    block = 0), for the record; None in Stochastic mode."""
    if w.mode != STRUCTURAL:
        return None
    if w.block > 0:
        return w.block
    b_max = max(1, min(w.N, (w.density_ppm * w.N + 500_000) // 1_000_000))
    return max(1, min(w.N // 10, b_max))


if __name__ == "__main__":
    main()
