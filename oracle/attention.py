"""Masked softmax attention over the unified index set (oracle; test only).

For query head h, row q and its KV head g = floor(h / G) (G = Hq / Hkv):

    s_j = scale * <Q[h, q], K[g, j]>        for j in I(g, q)
    p   = softmax(s)                        one normalisation over all of I
    out[h, q] = sum_j p_j V[g, j]

This is the paper's Pre-Fusion Unified Softmax (Methods, "Hybrid Anchor and
Pre-Fusion Unified Softmax"): every selected index -- local, global or
stochastic, from any seed -- enters one softmax exactly once; fragments are
never normalised apart and then combined.  The score and value products are
the paper's ``matmul_qk`` and ``matmul_av`` (Results, "Hardware Profiling")
restricted to the selected keys.

Reading: ``scale = 1/sqrt(D)`` (the paper is silent; it is the default of the
host models).  Arithmetic is float64 on the exact values of the inputs; the
max is subtracted before ``exp`` (softmax is invariant to it).
"""

import numpy as np


def sparse_attention(Q, K, V, row_ptr, col_idx, scale=None, rows=None):
    """out[Hq, N, D] (float64) from CSR sets; ``rows`` optionally restricts
    the computation to a list of (h, q) pairs and returns just those rows."""
    Q = np.asarray(Q)
    Hq, N, D = Q.shape
    Hkv = K.shape[0]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    if rows is None:
        rows = [(h, q) for h in range(Hq) for q in range(N)]
        out = np.zeros((Hq, N, D), dtype=np.float64)
        full = True
    else:
        out = np.zeros((len(rows), D), dtype=np.float64)
        full = False
    for t, (h, q) in enumerate(rows):
        g = h // G
        r = g * N + q
        idx = np.asarray(col_idx[row_ptr[r]:row_ptr[r + 1]], dtype=np.int64)
        o = attend_one(Q[h, q], K[g, idx], V[g, idx], scale)
        if full:
            out[h, q] = o
        else:
            out[t] = o
    return out


def attend_one(q, Ksel, Vsel, scale):
    """One row: softmax(scale * Ksel q) @ Vsel in float64."""
    q = np.asarray(q, dtype=np.float64)
    Ksel = np.asarray(Ksel, dtype=np.float64)
    Vsel = np.asarray(Vsel, dtype=np.float64)
    if Ksel.shape[0] == 0:
        return np.zeros(q.shape[-1], dtype=np.float64)
    s = (Ksel @ q) * scale
    p = np.exp(s - s.max())
    return (p @ Vsel) / p.sum()


def dense_causal(Q, K, V, scale=None):
    """Textbook dense causal softmax attention with GQA, float64 (for pins)."""
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    Hq, N, D = Q.shape
    G = Hq // K.shape[0]
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    out = np.empty_like(Q)
    tri = np.tril(np.ones((N, N), dtype=bool))
    for h in range(Hq):
        s = (Q[h] @ K[h // G].T) * scale
        s = np.where(tri, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        out[h] = (p @ V[h // G]) / p.sum(axis=1, keepdims=True)
    return out
