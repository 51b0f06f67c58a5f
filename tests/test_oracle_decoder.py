"""Pins of the decoder-layer oracle (the language model's layer over the
pruned input) to things other than itself: transformers' LLaMA decoder layer
(eager attention, float64) with the same weights, the residual form (zero
output projections give y = x), causality (a row's output does not depend on
later rows), the independence of packed sequences, and RMSNorm's and SiLU's
definitions."""
import math

import numpy as np
import pytest

from oracle.decoder import decoder_layer, rms_norm, silu


def _params(rng, d, ff, scale=0.2):
    return {"attn_norm": 1.0 + 0.1 * rng.standard_normal(d), "w_qkv": scale * rng.standard_normal((3 * d, d)),
            "w_o": scale * rng.standard_normal((d, d)), "ffn_norm": 1.0 + 0.1 * rng.standard_normal(d),
            "w_gate_up": scale * rng.standard_normal((2 * ff, d)), "w_down": scale * rng.standard_normal((d, ff))}


def test_rms_norm_and_silu_definitions():
    x = np.array([[3.0, 4.0]])
    np.testing.assert_allclose(rms_norm(x, np.array([1.0, 2.0]), 0.0), [[3 / math.sqrt(12.5), 8 / math.sqrt(12.5)]])
    np.testing.assert_allclose(silu(np.array([0.0, 1.0, -2.0])), [0.0, 1 / (1 + math.exp(-1)), -2 / (1 + math.exp(2))])


def test_matches_transformers_llama_decoder_layer():
    torch = pytest.importorskip("torch")
    llama = pytest.importorskip("transformers.models.llama.modeling_llama")
    from transformers import LlamaConfig
    # transformers' RMSNorm runs in float32 (about 1e-7 relative); eps is large
    # here so that a misplaced eps would show far above that
    d, H, ff, S, theta, eps = 32, 4, 48, 11, 10000.0, 0.05
    rng = np.random.default_rng(0)
    p = _params(rng, d, ff)
    X = rng.standard_normal((S, d))
    pos = np.array([0, 1, 3, 4, 9, 10, 12, 20, 21, 22, 23])   # kept visual tokens keep their indices
    cfg = LlamaConfig(hidden_size=d, num_attention_heads=H, num_key_value_heads=H, head_dim=d // H,
                      intermediate_size=ff, rms_norm_eps=eps, rope_theta=theta, attention_bias=False,
                      mlp_bias=False)
    cfg._attn_implementation = "eager"
    layer = llama.LlamaDecoderLayer(cfg, layer_idx=0).double()
    with torch.no_grad():
        layer.input_layernorm.weight.copy_(torch.tensor(p["attn_norm"]))
        layer.post_attention_layernorm.weight.copy_(torch.tensor(p["ffn_norm"]))
        layer.self_attn.q_proj.weight.copy_(torch.tensor(p["w_qkv"][:d]))
        layer.self_attn.k_proj.weight.copy_(torch.tensor(p["w_qkv"][d:2 * d]))
        layer.self_attn.v_proj.weight.copy_(torch.tensor(p["w_qkv"][2 * d:]))
        layer.self_attn.o_proj.weight.copy_(torch.tensor(p["w_o"]))
        layer.mlp.gate_proj.weight.copy_(torch.tensor(p["w_gate_up"][:ff]))
        layer.mlp.up_proj.weight.copy_(torch.tensor(p["w_gate_up"][ff:]))
        layer.mlp.down_proj.weight.copy_(torch.tensor(p["w_down"]))
        inv = 1.0 / (theta ** (torch.arange(0, d // H, 2, dtype=torch.float64) / (d // H)))
        ang = torch.tensor(pos, dtype=torch.float64)[:, None] * inv[None, :]
        cos = torch.cat([ang.cos()] * 2, dim=1)[None]
        sin = torch.cat([ang.sin()] * 2, dim=1)[None]
        mask = torch.full((S, S), -torch.inf, dtype=torch.float64).triu(1)[None, None]
        y = layer(torch.tensor(X)[None], attention_mask=mask, position_ids=torch.tensor(pos)[None],
                  position_embeddings=(cos, sin))
        y = y[0] if isinstance(y, tuple) else y
    want = y[0].numpy()
    got = decoder_layer(X, pos, [0, S], p, H, theta, eps)
    np.testing.assert_allclose(got, want, rtol=2e-5, atol=2e-6)
    assert np.max(np.abs(decoder_layer(X, pos, [0, S], p, H, theta, 1e-6) - want)) > 1e-3


def test_zero_projections_give_the_residual():
    rng = np.random.default_rng(1)
    p = _params(rng, 16, 24)
    p["w_o"][:] = 0.0
    p["w_down"][:] = 0.0
    X = rng.standard_normal((7, 16))
    np.testing.assert_array_equal(decoder_layer(X, np.arange(7), [0, 7], p, 2), X)


def test_causal_and_sequences_independent():
    rng = np.random.default_rng(2)
    p = _params(rng, 16, 24)
    X = rng.standard_normal((12, 16))
    pos = np.arange(12) * 2
    y = decoder_layer(X, pos, [0, 5, 12], p, 4)
    X2 = X.copy()
    X2[3:5] += 1.0                          # later rows of sequence 0
    y2 = decoder_layer(X2, pos, [0, 5, 12], p, 4)
    np.testing.assert_array_equal(y2[:3], y[:3])
    np.testing.assert_array_equal(y2[5:], y[5:])    # sequence 1 does not see sequence 0
    assert np.max(np.abs(y2[3:5] - y[3:5])) > 1e-3
    # each sequence alone gives the same rows
    np.testing.assert_allclose(decoder_layer(X[5:], pos[5:], [0, 7], p, 4), y[5:], rtol=1e-13, atol=1e-13)
