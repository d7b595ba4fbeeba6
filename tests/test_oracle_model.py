"""Pins for the oracle's model-level prefill (oracle/model.py).

At 100% density the RIS geometry of every row is its causal prefix, so the
stack must equal the host model's own dense implementation: the oracle is
checked against ``transformers``' Qwen2Model and LlamaModel (eager attention,
float64, the same random weights), with plain, linear and YaRN RoPE.
"""
from dataclasses import replace

import numpy as np
import pytest

from oracle import geometry as geo
from oracle import model as om
from oracle import rope
from synth import MODELS, model_weights, tokens

torch = pytest.importorskip("torch")
transformers = pytest.importorskip("transformers")
from transformers import LlamaConfig, LlamaModel, Qwen2Config, Qwen2Model  # noqa: E402


def hf_model(cfg, W, kind, s):
    params = {"rope_theta": cfg.rope_base}
    if kind == rope.PLAIN:
        params["rope_type"] = "default"
    elif kind == rope.LINEAR:
        params.update(rope_type="linear", factor=s)
    else:
        params.update(rope_type="yarn", factor=s, original_max_position_embeddings=cfg.native_len)
    common = dict(vocab_size=cfg.vocab, hidden_size=cfg.hidden, intermediate_size=cfg.inter,
                  num_hidden_layers=cfg.layers, num_attention_heads=cfg.heads,
                  num_key_value_heads=cfg.kv_heads, head_dim=cfg.head_dim, rms_norm_eps=cfg.eps,
                  max_position_embeddings=int(cfg.native_len * max(s, 1)), rope_parameters=params,
                  hidden_act="silu", tie_word_embeddings=False)
    if cfg.qkv_bias:
        conf = Qwen2Config(**common)
        cls = Qwen2Model
    else:
        conf = LlamaConfig(attention_bias=False, mlp_bias=False, **common)
        cls = LlamaModel
    conf._attn_implementation = "eager"
    m = cls(conf).double().eval()
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))  # noqa: E731
    with torch.no_grad():
        m.embed_tokens.weight.copy_(t(W["embed"]))
        for layer, L in zip(m.layers, W["layers"]):
            at = layer.self_attn
            at.q_proj.weight.copy_(t(L["q"]))
            at.k_proj.weight.copy_(t(L["k"]))
            at.v_proj.weight.copy_(t(L["v"]))
            if cfg.qkv_bias:
                at.q_proj.bias.copy_(t(L["bq"]))
                at.k_proj.bias.copy_(t(L["bk"]))
                at.v_proj.bias.copy_(t(L["bv"]))
            at.o_proj.weight.copy_(t(L["o"]))
            layer.mlp.gate_proj.weight.copy_(t(L["gate"]))
            layer.mlp.up_proj.weight.copy_(t(L["up"]))
            layer.mlp.down_proj.weight.copy_(t(L["down"]))
            layer.input_layernorm.weight.copy_(t(L["ln1"]))
            layer.post_attention_layernorm.weight.copy_(t(L["ln2"]))
        m.norm.weight.copy_(t(W["norm"]))
    return m


@pytest.mark.parametrize("name", ["tiny_qwen2", "tiny_llama"])
@pytest.mark.parametrize("kind,factor", [(rope.PLAIN, 1.0), (rope.LINEAR, 2.0), (rope.YARN, 2.0)])
def test_full_density_stack_equals_transformers(name, kind, factor):
    cfg = MODELS[name]
    W = model_weights(cfg, seed=3)
    N = 48
    ids = tokens(N, cfg.vocab, seed=4)
    spec = geo.MaskSpec(mode=geo.STOCHASTIC, density_ppm=10**6, seed=0, n_seeds=1, layer=0, N=N,
                        heads=cfg.kv_heads)
    got = om.prefill(ids, W, cfg, spec, kind, factor if kind != rope.PLAIN else 0.0)
    m = hf_model(cfg, W, kind, factor)
    with torch.no_grad():
        want = m(input_ids=torch.tensor(ids)[None]).last_hidden_state[0].numpy()
    # transformers computes the rotary frequencies in float32
    np.testing.assert_allclose(got, want, atol=2e-5, rtol=0)


def test_layers_use_distinct_geometries_and_sparsity_matters():
    """Layer l uses its own layer index in the hash, and at 5% density the
    stack differs from the dense one."""
    cfg = MODELS["tiny_qwen2"]
    N = 64
    spec = geo.MaskSpec(mode=geo.STOCHASTIC, density_ppm=50_000, seed=0, n_seeds=2, layer=0, N=N,
                        heads=cfg.kv_heads)
    a = geo.build_csr(replace(spec, layer=0))
    b = geo.build_csr(replace(spec, layer=1))
    assert not (np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]))
    W = model_weights(cfg, seed=1)
    ids = tokens(N, cfg.vocab, seed=2)
    sparse = om.prefill(ids, W, cfg, spec)
    dense = om.prefill(ids, W, cfg, replace(spec, density_ppm=10**6))
    assert np.abs(sparse - dense).max() > 1e-3
    assert np.isfinite(sparse).all()


def test_rmsnorm_and_silu_closed_forms():
    x = np.array([[3.0, 4.0], [0.0, 0.0]])
    w = np.array([2.0, 0.5])
    y = om.rmsnorm(x, w, 1e-6)
    r = np.sqrt(12.5 + 1e-6)
    np.testing.assert_allclose(y[0], [6.0 / r, 2.0 / r], rtol=1e-15)
    assert np.all(y[1] == 0)
    np.testing.assert_allclose(om.silu(np.array([0.0, 1.0])), [0.0, 1 / (1 + np.exp(-1.0))])
