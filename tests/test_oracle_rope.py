"""Pins for the oracle's RoPE (see oracle/rope.py).

The paper hands its factor to the Hugging Face configuration pathway, so the
transformers library's own RoPE initialisers and rotation are independent
implementations of what the paper ran.
"""
import math

import numpy as np
import pytest
import torch

from oracle import rope

transformers = pytest.importorskip("transformers")
from transformers import Qwen2Config  # noqa: E402
from transformers.modeling_rope_utils import ROPE_INIT_FUNCTIONS  # noqa: E402
from transformers.models.llama.modeling_llama import apply_rotary_pos_emb  # noqa: E402
from transformers.models.qwen2.modeling_qwen2 import Qwen2RotaryEmbedding  # noqa: E402


def hf_config(D, base, kind, s=1.0, orig=32768, heads=12):
    params = {"rope_theta": base}
    if kind == rope.PLAIN:
        params["rope_type"] = "default"
    elif kind == rope.LINEAR:
        params.update(rope_type="linear", factor=s)
    else:
        params.update(rope_type="yarn", factor=s, original_max_position_embeddings=orig)
    return Qwen2Config(hidden_size=D * heads, num_attention_heads=heads, head_dim=D,
                       max_position_embeddings=int(orig * max(s, 1)), rope_parameters=params)


CASES = [
    (128, 1e6, rope.PLAIN, 1.0, 32768),
    (128, 1e6, rope.LINEAR, 2.0, 32768),
    (128, 1e6, rope.YARN, 2.0, 32768),      # Qwen2 at 65,536 tokens
    (64, 1e4, rope.YARN, 32.0, 2048),       # TinyLlama at 65,536 tokens
    (64, 1e4, rope.YARN, 4.0, 2048),
    (128, 1e6, rope.LINEAR, 4.0, 32768),
]


@pytest.mark.parametrize("D,base,kind,s,orig", CASES)
def test_inv_freq_and_mscale_match_transformers(D, base, kind, s, orig):
    cfg = hf_config(D, base, kind, s, orig)
    if kind == rope.PLAIN:
        emb = Qwen2RotaryEmbedding(cfg)
        want, att = emb.inv_freq.double().numpy(), emb.attention_scaling
    else:
        inv, att = ROPE_INIT_FUNCTIONS["linear" if kind == rope.LINEAR else "yarn"](cfg, None)
        want = inv.double().numpy()
    got = rope.inv_freq(kind, D, base, s, orig)
    np.testing.assert_allclose(got, want, rtol=2e-6)        # transformers works in float32
    assert rope.mscale(kind, s) == pytest.approx(att, rel=1e-12)


def test_yarn_frequency_bands_qwen2():
    """Qwen2 (D = 128, base 1e6, native 32,768) at 2x: the correction range is
    [floor(23.6), ceil(39.65)] = [23, 40]; below it frequencies are kept, above
    it they are divided by s; mscale = 0.1 ln 2 + 1."""
    f = rope.inv_freq(rope.YARN, 128, 1e6, 2.0, 32768)
    plain = rope.inv_freq(rope.PLAIN, 128, 1e6)
    np.testing.assert_array_equal(f[:24], plain[:24])
    np.testing.assert_allclose(f[40:], plain[40:] / 2.0, rtol=1e-15)
    assert np.all((f[24:40] < plain[24:40]) & (f[24:40] > plain[24:40] / 2))
    assert rope.mscale(rope.YARN, 2.0) == pytest.approx(1.0693147180559945)
    assert rope.mscale(rope.YARN, 32.0) == pytest.approx(1.3465735902799727)


def test_rotation_matches_transformers_apply_rotary_pos_emb():
    rng = np.random.default_rng(0)
    D, N = 128, 64
    x = rng.standard_normal((2, N, D))
    for kind, s in [(rope.PLAIN, 1.0), (rope.YARN, 2.0), (rope.LINEAR, 3.0)]:
        pos0 = 1000
        got = rope.apply(x, kind, 1e6, pos0=pos0, s=s, orig_max_pos=32768)
        c, sn = rope.cos_sin(kind, D, 1e6, np.arange(pos0, pos0 + N), s, 32768)
        cos = torch.from_numpy(np.concatenate([c, c], axis=-1))[None]
        sin = torch.from_numpy(np.concatenate([sn, sn], axis=-1))[None]
        xt = torch.from_numpy(x)[None]
        qe, _ = apply_rotary_pos_emb(xt, xt, cos, sin, unsqueeze_dim=1)
        np.testing.assert_allclose(got, qe[0].numpy(), rtol=0, atol=1e-12)


def test_cos_sin_match_transformers_rotary_embedding_forward():
    """End-to-end against the model's rotary module (float32, small positions)."""
    for kind, s in [(rope.PLAIN, 1.0), (rope.YARN, 2.0)]:
        cfg = hf_config(128, 1e6, kind, s, 32768)
        emb = Qwen2RotaryEmbedding(cfg)
        pos = torch.arange(0, 512)[None]
        cos, sin = emb(torch.zeros(1, 512, 128), pos)
        c, sn = rope.cos_sin(kind, 128, 1e6, np.arange(512), s, 32768)
        np.testing.assert_allclose(cos[0, :, :64].double().numpy(), c, atol=2e-4)
        np.testing.assert_allclose(sin[0, :, 64:].double().numpy(), sn, atol=2e-4)


def test_relative_position_and_norm_invariants():
    rng = np.random.default_rng(1)
    D = 64
    x = rng.standard_normal((1, 1, D))
    y = rng.standard_normal((1, 1, D))
    for kind, s in [(rope.PLAIN, 1.0), (rope.YARN, 4.0), (rope.LINEAR, 2.0)]:
        ms = rope.mscale(kind, s)
        dots = []
        for m, n in [(5, 2), (1005, 1002), (60003, 60000)]:
            a = rope.apply(x, kind, 1e4, pos0=m, s=s, orig_max_pos=2048)
            b = rope.apply(y, kind, 1e4, pos0=n, s=s, orig_max_pos=2048)
            dots.append(float(np.sum(a * b)))
            assert np.linalg.norm(a) == pytest.approx(ms * np.linalg.norm(x), rel=1e-12)
        assert dots[0] == pytest.approx(dots[1], rel=1e-9, abs=1e-9)
        assert dots[0] == pytest.approx(dots[2], rel=1e-8, abs=1e-8)


def test_linear_is_position_compression_and_unit_yarn_is_plain():
    D = 128
    p = np.arange(0, 4000, 7, dtype=np.float64)
    c_lin, s_lin = rope.cos_sin(rope.LINEAR, D, 1e6, p, 2.0)
    c_pl, s_pl = rope.cos_sin(rope.PLAIN, D, 1e6, p / 2.0)
    np.testing.assert_allclose(c_lin, c_pl, atol=1e-12)
    np.testing.assert_allclose(s_lin, s_pl, atol=1e-12)
    f1 = rope.inv_freq(rope.YARN, D, 1e6, 1.0, 32768)
    np.testing.assert_allclose(f1, rope.inv_freq(rope.PLAIN, D, 1e6), rtol=1e-15)
    assert rope.mscale(rope.YARN, 1.0) == 1.0


def test_scale_factor_is_window_over_native_limit():
    assert rope.scale_factor(0, 65536, 32768) == 2.0
    assert rope.scale_factor(0, 32768, 32768) == 1.0
    assert rope.scale_factor(0, 1000, 32768) == 1.0
    assert rope.scale_factor(0, 65536, 2048) == 32.0
    assert rope.scale_factor(3.0, 65536, 32768) == 3.0
    assert math.isclose(rope.scale_factor(0, 50000, 32768), 50000 / 32768)
