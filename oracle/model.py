"""Model-level prefill through a decoder stack with RIS attention (oracle;
TEST INFRASTRUCTURE ONLY).

The paper swaps only the attention of a LLaMA- or Qwen2-architecture model;
weights, tokenizer and every other layer stay as they are (Methods, opening
of "The RIS Implementation").  This module is that host stack written out in
float64: per layer

    h = RMSNorm(x) ; q, k, v = h Wq^T (+ bq), h Wk^T (+ bk), h Wv^T (+ bv)
    q, k <- RoPE (the model's base, the paper's scaling; Methods,
            "Dynamic RoPE Scaling")
    a = sparse attention over the RIS geometry of this layer (PFUS)
    x = x + a Wo^T
    h = RMSNorm(x) ; x = x + (silu(h Wg^T) * (h Wu^T)) Wd^T

followed by a final RMSNorm, RMSNorm(x) = x / sqrt(mean(x^2) + eps) * w.
Layer l uses the geometry descriptor with its own layer index (distinct sets
per layer).  No LM head: the stack returns the final hidden states.
"""

from dataclasses import replace

import numpy as np

from . import attention, geometry, rope


def rmsnorm(x, w, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * np.asarray(w, dtype=np.float64)


def silu(x):
    return x / (1.0 + np.exp(-x))


def attention_block(h, L, cfg, spec, rope_kind, rope_factor):
    """Attention sublayer on normalised input h [N, hidden]; returns [N, hidden]."""
    N = h.shape[0]
    D = cfg.head_dim

    def proj(name):
        y = h @ np.asarray(L[name], dtype=np.float64).T
        if cfg.qkv_bias:
            y = y + np.asarray(L["b" + name], dtype=np.float64)
        return y

    q = proj("q").reshape(N, cfg.heads, D).transpose(1, 0, 2)
    k = proj("k").reshape(N, cfg.kv_heads, D).transpose(1, 0, 2)
    v = proj("v").reshape(N, cfg.kv_heads, D).transpose(1, 0, 2)
    if rope_kind is not None:
        s = rope.scale_factor(rope_factor, N, cfg.native_len) if rope_kind != rope.PLAIN else 1.0
        q = rope.apply(q, rope_kind, cfg.rope_base, 0, s, cfg.native_len)
        k = rope.apply(k, rope_kind, cfg.rope_base, 0, s, cfg.native_len)
    row_ptr, col_idx = geometry.build_csr(spec)
    a = attention.sparse_attention(q, k, v, row_ptr, col_idx)        # [Hq, N, D]
    a = a.transpose(1, 0, 2).reshape(N, cfg.heads * D)
    return a @ np.asarray(L["o"], dtype=np.float64).T


def mlp_block(h, L):
    g = h @ np.asarray(L["gate"], dtype=np.float64).T
    u = h @ np.asarray(L["up"], dtype=np.float64).T
    return (silu(g) * u) @ np.asarray(L["down"], dtype=np.float64).T


def prefill(tokens, W, cfg, spec, rope_kind=rope.PLAIN, rope_factor=0.0):
    """Final hidden states [N, hidden] of the stack for token ids ``tokens``.

    spec: the geometry descriptor (``geometry.MaskSpec``, heads = kv_heads,
    N = len(tokens)); layer l uses ``replace(spec, layer=l)``.  rope_kind:
    ``rope.PLAIN``, ``rope.LINEAR``, ``rope.YARN`` or None (no rotation);
    rope_factor 0 takes the window / native-limit rule.
    """
    x = np.asarray(W["embed"], dtype=np.float64)[np.asarray(tokens)]
    for l, L in enumerate(W["layers"]):
        x = x + attention_block(rmsnorm(x, L["ln1"], cfg.eps), L, cfg, replace(spec, layer=l), rope_kind,
                                rope_factor)
        x = x + mlp_block(rmsnorm(x, L["ln2"], cfg.eps), L)
    return rmsnorm(x, W["norm"], cfg.eps)
