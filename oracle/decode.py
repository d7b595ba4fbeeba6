"""Hybrid-Anchor decode step (oracle; TEST INFRASTRUCTURE ONLY).

Methods, "Hybrid Anchor and Pre-Fusion Unified Softmax": during generation
the index set has two parts with different update rates.  When the first
token is generated (position ``t0``) the union of every seed's indices for
that row is computed once and frozen -- the *Stochastic Anchor*.  Every later
step recomputes only a *Dynamic Local Window* over the most recent tokens.
The two merge through ``unique()`` before K/V extraction and feed one
softmax (PFUS).

Readings (also in the design notes):

1. The anchor of KV head g is the prefill geometry's row ``t0`` (the draws of
   every seed, plus the Structural clique) without the window and the
   initial-token range: those are recomputed per step.
2. At step position ``t`` the set is
   ``unique(anchor U [max(0, t - L + 1), t] U [0, min(A, t + 1)))``; with
   ``L = 0`` there is no window.  Anchor entries are all ``<= t0 <= t``.
3. At ``t = t0`` the step set equals the full prefill geometry's row ``t0``
   (window L and anchor A included) -- the two definitions agree on the first
   generated token.
"""

from dataclasses import replace

import numpy as np

from . import attention, geometry


def stochastic_anchor(spec, kv_head, t0):
    """The frozen union for KV head ``kv_head`` at the first generated
    position ``t0`` (reading 1); ascending, unique."""
    if not 0 <= t0 < spec.N:
        raise ValueError("t0 must lie in [0, N)")
    return geometry.row_set(replace(spec, window=0, anchor=0), kv_head, t0)


def step_set(anchor, t, window, sink):
    """Indices attended at position ``t`` (reading 2): the frozen anchor, the
    local window of ``window`` tokens ending at ``t`` and the first ``sink``
    tokens, merged with ``unique``."""
    anchor = np.asarray(anchor, dtype=np.int64)
    parts = [anchor[anchor <= t]]
    if window > 0:
        parts.append(np.arange(max(0, t - window + 1), t + 1, dtype=np.int64))
    if sink > 0:
        parts.append(np.arange(0, min(sink, t + 1), dtype=np.int64))
    return np.unique(np.concatenate(parts))


def decode_attention(q, K, V, idx, scale):
    """One generated token: q [G, D] (the G query heads of one KV group),
    K, V [T, D] the group's cache; one softmax over ``idx`` per head."""
    out = np.zeros((q.shape[0], V.shape[1]), dtype=np.float64)
    if len(idx) == 0:
        return out
    for h in range(q.shape[0]):
        out[h] = attention.attend_one(q[h], K[idx], V[idx], scale)
    return out
