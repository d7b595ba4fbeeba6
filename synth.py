"""Seeded synthetic inputs for RIS sparse attention.

This module only *makes inputs*: Gaussian Q/K/V at the layer shapes of the
paper's host models, the bf16 rounding of those inputs, and the planted
"needle" similarities of the Structural workload.  It holds none of the
method's arithmetic (no hash, draw, RoPE or softmax) and is the only code that
both the CPU oracle's tests and the GPU path's tests use.

The paper evaluates on concatenated scientific manuscripts and QA sets with
trained Qwen2-1.5B / TinyLlama-1.1B weights; none of those are available, so
Gaussian activations of the same shapes stand in for them (Results,
"Empirical Evaluation"; Discussion, "Hardware Context").
"""

from dataclasses import dataclass, replace

import numpy as np

STOCHASTIC, STRUCTURAL = 0, 1
ROPE_NONE, ROPE_PLAIN, ROPE_LINEAR, ROPE_YARN = -1, 0, 1, 2


@dataclass(frozen=True)
class Workload:
    name: str
    Hq: int
    Hkv: int
    D: int
    N: int
    dtype: str                 # "f32" or "bf16" (input element type)
    mode: int
    density_ppm: int
    n_seeds: int
    block: int = 0             # Structural block size (0 = paper rule)
    rope: int = ROPE_NONE
    rope_base: float = 10000.0
    rope_orig: int = 0         # native positional limit
    rope_factor: float = 0.0   # 0 = window / native limit
    layers: int = 1
    needles: bool = False
    seed: int = 0              # first ensemble seed
    window: int = 0            # dense local window L (0 = none)
    anchor: int = 0            # initial-token anchor A (0 = none)

    def scaled(self, N):
        return replace(self, N=N)


# The five workloads: a tiny fp32 case, Qwen2-1.5B-shaped layers (12 query /
# 2 KV heads, head_dim 128) at 32k and 64k tokens, and a TinyLlama-1.1B-shaped
# layer (32 / 4 heads, head_dim 64) at 64k tokens over 22 layers.
WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 64, 512, "f32", STOCHASTIC, 100_000, 1),
    "qwen2_32k_stochastic": Workload(
        "qwen2_32k_stochastic", 12, 2, 128, 32768, "bf16", STOCHASTIC, 10_000, 10,
        rope=ROPE_PLAIN, rope_base=1e6, rope_orig=32768),
    "qwen2_32k_structural": Workload(
        "qwen2_32k_structural", 12, 2, 128, 32768, "bf16", STRUCTURAL, 10_000, 10,
        block=64, rope=ROPE_PLAIN, rope_base=1e6, rope_orig=32768, needles=True),
    "qwen2_64k_stochastic_yarn": Workload(
        "qwen2_64k_stochastic_yarn", 12, 2, 128, 65536, "bf16", STOCHASTIC, 10_000, 70,
        rope=ROPE_YARN, rope_base=1e6, rope_orig=32768),
    "tinyllama_64k_structural": Workload(
        "tinyllama_64k_structural", 32, 4, 64, 65536, "bf16", STRUCTURAL, 50_000, 10,
        block=64, layers=22),
    # The 64k Qwen2 layer with the paper's full geometry: the 70-seed ensemble
    # plus a dense local window of 1,024 tokens and an anchor of 4 initial
    # tokens (the paper gives no anchor size).
    "qwen2_64k_full_geometry": Workload(
        "qwen2_64k_full_geometry", 12, 2, 128, 65536, "bf16", STOCHASTIC, 10_000, 70,
        rope=ROPE_YARN, rope_base=1e6, rope_orig=32768, window=1024, anchor=4),
    # The Structural workloads with the paper's own block rule,
    # B = min(floor(N / 10), round(d N)): B = 328 at 32k / 1%, 3,277 at
    # 64k / 5% (one layer).
    "qwen2_32k_structural_paper_block": Workload(
        "qwen2_32k_structural_paper_block", 12, 2, 128, 32768, "bf16", STRUCTURAL, 10_000, 10,
        block=0, rope=ROPE_PLAIN, rope_base=1e6, rope_orig=32768),
    "tinyllama_64k_structural_paper_block": Workload(
        "tinyllama_64k_structural_paper_block", 32, 4, 64, 65536, "bf16", STRUCTURAL, 50_000, 10,
        block=0),
}


def gaussian_qkv(Hq, Hkv, N, D, seed=0):
    """Q [Hq,N,D], K [Hkv,N,D], V [Hkv,N,D] ~ N(0,1) float32, drawn in that
    order from ``numpy.random.default_rng(seed)``."""
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((Hq, N, D), dtype=np.float32)
    K = rng.standard_normal((Hkv, N, D), dtype=np.float32)
    V = rng.standard_normal((Hkv, N, D), dtype=np.float32)
    return Q, K, V


def to_bf16(x):
    """Round a float32 array to bfloat16 (round to nearest even).

    Returns a torch.bfloat16 CPU tensor; ``.float().numpy()`` gives the exact
    values it holds.
    """
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)


def needle_plan(N, seed=1, span=512, per_span=8, targets=64):
    """Needle positions and their target queries.

    In every ``span``-token window ``per_span`` key positions p are chosen;
    for each p, ``targets`` query rows are chosen uniformly without
    replacement from [p, N) (all of them if fewer remain).  Returns arrays
    (p, i) of equal length.
    """
    rng = np.random.default_rng(seed)
    ps, iss = [], []
    for s0 in range(0, N, span):
        width = min(span, N - s0)
        pos = s0 + rng.choice(width, size=min(per_span, width), replace=False)
        for p in np.sort(pos):
            avail = N - p
            t = rng.choice(avail, size=min(targets, avail), replace=False) + p
            ps.append(np.full(t.shape, p, dtype=np.int64))
            iss.append(t.astype(np.int64))
    return np.concatenate(ps), np.concatenate(iss)


def plant_needles(Q, K, plan, sigma_mult=3.0):
    """Raise <Q[h,i], K[g,p]> by sigma_mult * sqrt(D) for every planned (p, i)
    and every query head h of KV group g.

    Q: [Hq,N,D] float array (modified copy returned), K: [Hkv,N,D].  Applied
    to rotated (post-RoPE) vectors, so the logit gain is exact.
    """
    Q = np.array(Q, dtype=np.float64, copy=True)
    K = np.asarray(K, dtype=np.float64)
    Hq, N, D = Q.shape
    Hkv = K.shape[0]
    G = Hq // Hkv
    p, i = plan
    for g in range(Hkv):
        kp = K[g, p]                                          # [P, D]
        add = sigma_mult * np.sqrt(D) * kp / np.sum(kp * kp, axis=1, keepdims=True)
        for h in range(g * G, (g + 1) * G):
            np.add.at(Q[h], i, add)
    return Q


def decode_inputs(B, Hq, Hkv, max_len, D, seed=0):
    """Decode-step inputs ~ N(0,1) float32, drawn in this order from
    ``numpy.random.default_rng(seed)``: the new tokens' queries Q [B, Hq, D]
    and the caches K, V [B, Hkv, max_len, D]."""
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((B, Hq, D), dtype=np.float32)
    K = rng.standard_normal((B, Hkv, max_len, D), dtype=np.float32)
    V = rng.standard_normal((B, Hkv, max_len, D), dtype=np.float32)
    return Q, K, V


# ---------------------------------------------------------------------------
# Host-model shapes for a model-level prefill with random weights.
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelConfig:
    name: str
    hidden: int
    heads: int
    kv_heads: int
    head_dim: int
    inter: int                 # MLP intermediate size
    layers: int
    eps: float                 # RMSNorm epsilon
    rope_base: float
    qkv_bias: bool             # Qwen2 has q/k/v biases, LLaMA does not
    vocab: int
    native_len: int            # positional limit the model was trained to

    def with_layers(self, n):
        return replace(self, layers=n)


MODELS = {
    "qwen2_1.5b": ModelConfig("qwen2_1.5b", 1536, 12, 2, 128, 8960, 28, 1e-6, 1e6, True, 151936, 32768),
    "tinyllama_1.1b": ModelConfig("tinyllama_1.1b", 2048, 32, 4, 64, 5632, 22, 1e-5, 1e4, False, 32000,
                                  2048),
    # small stand-ins with the same layer structure, for parity tests
    "tiny_qwen2": ModelConfig("tiny_qwen2", 256, 4, 2, 64, 512, 2, 1e-6, 1e6, True, 500, 128),
    "tiny_llama": ModelConfig("tiny_llama", 384, 6, 2, 64, 640, 2, 1e-5, 1e4, False, 500, 128),
}


def model_weights(cfg, seed=0):
    """Random weights of a decoder stack, float32, from
    ``numpy.random.default_rng(seed)`` in a fixed order: embedding, then per
    layer q, k, v (+ biases), o, gate, up, down and the two norm weights, then
    the final norm.  Linear weights and embeddings ~ N(0, 0.02^2), biases
    ~ N(0, 0.02^2), norm weights ~ 1 + N(0, 0.1^2).  Linear weights are stored
    [out_features, in_features]."""
    rng = np.random.default_rng(seed)
    f = np.float32

    def lin(o, i):
        return (0.02 * rng.standard_normal((o, i))).astype(f)

    W = {"embed": (0.02 * rng.standard_normal((cfg.vocab, cfg.hidden))).astype(f), "layers": []}
    qd, kd = cfg.heads * cfg.head_dim, cfg.kv_heads * cfg.head_dim
    for _ in range(cfg.layers):
        L = {"q": lin(qd, cfg.hidden), "k": lin(kd, cfg.hidden), "v": lin(kd, cfg.hidden)}
        if cfg.qkv_bias:
            L["bq"] = (0.02 * rng.standard_normal(qd)).astype(f)
            L["bk"] = (0.02 * rng.standard_normal(kd)).astype(f)
            L["bv"] = (0.02 * rng.standard_normal(kd)).astype(f)
        L["o"] = lin(cfg.hidden, qd)
        L["gate"] = lin(cfg.inter, cfg.hidden)
        L["up"] = lin(cfg.inter, cfg.hidden)
        L["down"] = lin(cfg.hidden, cfg.inter)
        L["ln1"] = (1 + 0.1 * rng.standard_normal(cfg.hidden)).astype(f)
        L["ln2"] = (1 + 0.1 * rng.standard_normal(cfg.hidden)).astype(f)
        W["layers"].append(L)
    W["norm"] = (1 + 0.1 * rng.standard_normal(cfg.hidden)).astype(f)
    return W


def tokens(n, vocab, seed=0):
    """n token ids uniform in [0, vocab) from ``default_rng(seed)``."""
    return np.random.default_rng(seed).integers(0, vocab, size=n)
