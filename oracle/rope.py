"""RoPE with the paper's long-context scaling (oracle; test infrastructure only).

The paper (Methods, "Dynamic RoPE Scaling") sets the RoPE factor at load time
to requested window / native limit and passes it through the Hugging Face
configuration pathway, which offers linear interpolation and YaRN (Results,
"Linear Interpolation" and "YaRN").  The frequencies here are therefore the
ones that pathway defines, written out in float64:

* plain:  inv_freq_i = base^(-2i/D),  i = 0 .. D/2 - 1
* linear: inv_freq_i / s  (positions compressed uniformly by s)
* YaRN (Peng et al., 2023, as released): with correction dimension
  ``cd(r) = D * ln(L_orig / (2 pi r)) / (2 ln base)``,
  ``low = max(floor(cd(beta_fast)), 0)``, ``high = min(ceil(cd(beta_slow)), D-1)``,
  ramp ``t_i = clamp((i - low) / (high - low), 0, 1)`` and
  ``inv_freq_i = t_i * base^(-2i/D) / s + (1 - t_i) * base^(-2i/D)``;
  cos and sin are multiplied by ``mscale = 0.1 ln s + 1`` (1 when s <= 1).

Rotation follows the half-split pairing of those models: dimension i pairs with
i + D/2, ``y_i = x_i cos - x_{i+D/2} sin`` and
``y_{i+D/2} = x_{i+D/2} cos + x_i sin`` at angle ``(pos0 + t) * inv_freq_i``.
Angles, cos and sin are float64 (the paper is silent; float32 angles at
position 65,535 would be off by ~4e-3 rad).

Pinned by: inverse frequencies and attention factor against the transformers
library's own RoPE initialisers; the rotation against transformers'
``apply_rotary_pos_emb``; invariants (relative-position dependence, norm times
mscale, linear(s) at p equals plain at p / s).
"""

import math

import numpy as np

PLAIN = 0
LINEAR = 1
YARN = 2


def scale_factor(factor, window, orig_max_pos):
    """The paper's factor: requested window / native limit, never below 1,
    unless an explicit factor (> 0) is given."""
    if factor and factor > 0:
        return float(factor)
    return max(1.0, float(window) / float(orig_max_pos))


def inv_freq(kind, D, base, s=1.0, orig_max_pos=None, beta_slow=1.0, beta_fast=32.0):
    """Inverse frequencies (float64, length D/2) for the given scaling."""
    i = np.arange(D // 2, dtype=np.float64)
    plain = 1.0 / np.power(float(base), 2.0 * i / D)
    if kind == PLAIN:
        return plain
    if kind == LINEAR:
        return plain / s
    if kind == YARN:
        def cd(rot):
            return (D * math.log(orig_max_pos / (rot * 2.0 * math.pi))) / (2.0 * math.log(base))
        low = max(math.floor(cd(beta_fast)), 0)
        high = min(math.ceil(cd(beta_slow)), D - 1)
        if low == high:
            high += 0.001
        ramp = np.clip((i - low) / (high - low), 0.0, 1.0)
        return ramp * (plain / s) + (1.0 - ramp) * plain
    raise ValueError(f"unknown RoPE kind {kind}")


def mscale(kind, s):
    """Attention (cos/sin) factor: 0.1 ln s + 1 for YaRN with s > 1, else 1."""
    if kind == YARN and s > 1.0:
        return 0.1 * math.log(s) + 1.0
    return 1.0


def cos_sin(kind, D, base, positions, s=1.0, orig_max_pos=None, beta_slow=1.0, beta_fast=32.0):
    """float64 (cos, sin) * mscale, shape (len(positions), D/2)."""
    f = inv_freq(kind, D, base, s, orig_max_pos, beta_slow, beta_fast)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * f[None, :]
    ms = mscale(kind, s)
    return np.cos(ang) * ms, np.sin(ang) * ms


def apply(x, kind, base, pos0=0, s=1.0, orig_max_pos=None, beta_slow=1.0, beta_fast=32.0,
          positions=None):
    """Rotate x [heads, N, D] (any float dtype) in float64; returns float64.

    Token t sits at position pos0 + t, or at positions[t] when given.
    """
    x = np.asarray(x, dtype=np.float64)
    H, N, D = x.shape
    pos = np.arange(pos0, pos0 + N) if positions is None else np.asarray(positions)
    c, sn = cos_sin(kind, D, base, pos, s, orig_max_pos, beta_slow, beta_fast)
    x1, x2 = x[..., : D // 2], x[..., D // 2:]
    return np.concatenate([x1 * c - x2 * sn, x2 * c + x1 * sn], axis=-1)
