"""Pins of the predictor oracle (Eq. (3)) to things other than itself:
textbook normal-CDF values, closed-form rotations, invariants the equation
implies, and independent library implementations (torch Linear / GELU /
scaled-dot-product attention, the LLaMA rotary embedding of transformers)."""
import math

import numpy as np
import pytest

from oracle import gelu_erf, mlp, predicted_attention, rope

# Standard normal CDF, textbook table values.
PHI_1 = 0.8413447460685429
PHI_2 = 0.9772498680518208
PHI_M1 = 0.15865525393145707


def test_gelu_textbook_values():
    got = gelu_erf(np.array([1.0, 2.0, -1.0, 0.0]))
    want = np.array([PHI_1, 2 * PHI_2, -PHI_M1, 0.0])
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)
    # the tanh approximation would be off by ~1.5e-4 at x = 1
    assert abs(got[0] - 0.8411919906082768) > 1e-4


def test_rope_two_dim_rotation_closed_form():
    for p in [0, 1, 2, 7, 100]:
        np.testing.assert_allclose(rope(np.array([[1.0, 0.0]]), np.array([p]), 1e4)[0],
                                   [math.cos(p), math.sin(p)], atol=1e-15)
        np.testing.assert_allclose(rope(np.array([[0.0, 1.0]]), np.array([p]), 1e4)[0],
                                   [-math.sin(p), math.cos(p)], atol=1e-15)


def test_rope_frequency_spectrum():
    # width 4, base 1e4: pair (0, 2) turns 1 rad / position, pair (1, 3) 0.01 rad.
    x = np.zeros((1, 4)); x[0, 1] = 1.0
    out = rope(x, np.array([100]), 1e4)[0]
    np.testing.assert_allclose(out, [0.0, math.cos(1.0), 0.0, math.sin(1.0)], atol=1e-14)


def test_rope_relative_position_property():
    rng = np.random.default_rng(0)
    q = rng.standard_normal((1, 16)); k = rng.standard_normal((1, 16))
    base = (rope(q, np.array([9]), 1e4) @ rope(k, np.array([4]), 1e4).T).item()
    for shift in [1, 17, 1000]:
        val = (rope(q, np.array([9 + shift]), 1e4) @ rope(k, np.array([4 + shift]), 1e4).T).item()
        assert abs(val - base) < 1e-12
    np.testing.assert_allclose(np.linalg.norm(rope(q, np.array([123]), 1e4)), np.linalg.norm(q))


def test_rope_matches_llama_rotary_embedding():
    torch = pytest.importorskip("torch")
    llama = pytest.importorskip("transformers.models.llama.modeling_llama")
    from transformers import LlamaConfig
    d, theta = 16, 10000.0
    cfg = LlamaConfig(hidden_size=d, num_attention_heads=1, head_dim=d, rope_theta=theta,
                      max_position_embeddings=4096)
    emb = llama.LlamaRotaryEmbedding(cfg)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, d))
    pos = np.array([0, 1, 5, 31, 63])
    cos, sin = emb(torch.zeros(1, 5, d), torch.tensor(pos)[None])
    xt = torch.tensor(x)[None, None]                       # [1, heads, seq, d]
    q_rot, _ = llama.apply_rotary_pos_emb(xt, xt, cos.double(), sin.double())
    # transformers builds its angles in float32; at positions < 64 that is ~1e-5 rad.
    np.testing.assert_allclose(rope(x, pos, theta), q_rot[0, 0].numpy(), atol=5e-5)


def _weights(rng, D, H, dp, scale=0.3):
    g = lambda *s: scale * rng.standard_normal(s)
    return {"w1_v": g(H, D), "b1_v": g(H), "w2_v": g(H, H), "b2_v": g(H), "w_k": g(dp, H),
            "w1_t": g(H, D), "b1_t": g(H), "w2_t": g(H, H), "b2_t": g(H), "w_q": g(dp, H)}


def _case(seed=0, N=37, M=5, D=24, H=16, dp=8):
    rng = np.random.default_rng(seed)
    V = rng.standard_normal((N, D)); T = rng.standard_normal((M, D))
    return V, T, np.arange(N), N + np.arange(M), _weights(rng, D, H, dp)


def test_p_hat_is_a_distribution():
    V, T, pv, pt, w = _case()
    p = predicted_attention(V, T, pv, pt, w)
    assert np.all(p > 0)
    assert abs(p.sum() - 1.0) < 1e-14


def test_zero_query_projection_gives_uniform():
    V, T, pv, pt, w = _case()
    w["w_q"] = np.zeros_like(w["w_q"])
    p = predicted_attention(V, T, pv, pt, w)
    np.testing.assert_allclose(p, 1.0 / V.shape[0], rtol=0, atol=1e-17)


def test_position_shift_invariance():
    V, T, pv, pt, w = _case()
    p0 = predicted_attention(V, T, pv, pt, w)
    p1 = predicted_attention(V, T, pv + 1000, pt + 1000, w)
    np.testing.assert_allclose(p1, p0, rtol=1e-10)


def test_permutation_equivariance():
    V, T, pv, pt, w = _case()
    perm = np.random.default_rng(3).permutation(V.shape[0])
    p0 = predicted_attention(V, T, pv, pt, w)
    p1 = predicted_attention(V[perm], T, pv[perm], pt, w)
    np.testing.assert_allclose(p1, p0[perm], rtol=1e-12)


def test_worked_example_softmax_then_mean():
    """Two-wide identity predictor at position 0 (RoPE is then the identity):
    keys are GELU of the visual rows, queries GELU of the question rows, so
    every value follows from the normal-CDF table.  Rows v = (0,0), (1,0),
    (2,0) give keys (0, Phi(1), 2 Phi(2)) on the first axis; questions
    (1,0) and (0,0) give queries Phi(1) and 0.  Query 1's logits are
    Phi(1) * key / sqrt(2); query 2's are all zero (uniform row)."""
    I2 = np.eye(2); z = np.zeros(2)
    w = {"w1_v": I2, "b1_v": z, "w2_v": I2, "b2_v": z, "w_k": I2,
         "w1_t": I2, "b1_t": z, "w2_t": I2, "b2_t": z, "w_q": I2}
    V = np.array([[0.0, 0.0], [1.0, 0.0], [2.0, 0.0]])
    T = np.array([[1.0, 0.0], [0.0, 0.0]])
    p = predicted_attention(V, T, np.zeros(3, int), np.zeros(2, int), w)
    logits = [0.0, PHI_1 * PHI_1 / math.sqrt(2), PHI_1 * 2 * PHI_2 / math.sqrt(2)]
    e = [math.exp(x) for x in logits]
    want = [0.5 * (ei / sum(e) + 1.0 / 3.0) for ei in e]
    np.testing.assert_allclose(p, want, rtol=1e-13)
    # averaging the logits before one softmax (the superseded form) differs:
    mean_logits = [0.5 * x for x in logits]
    em = [math.exp(x) for x in mean_logits]
    assert abs(p[2] - em[2] / sum(em)) > 1e-3


def test_predictor_matches_torch_modules():
    """f_V / f_T as torch Linear + exact GELU, scores through torch's
    scaled_dot_product_attention with the identity as values (its output rows
    are then the attention probabilities), positions 0..M-1 and N.. through
    the LLaMA rotary embedding."""
    torch = pytest.importorskip("torch")
    llama = pytest.importorskip("transformers.models.llama.modeling_llama")
    from transformers import LlamaConfig
    F = torch.nn.functional
    V, T, pv, pt, w = _case(seed=5, N=29, M=4, D=20, H=12, dp=8)
    pt = np.arange(T.shape[0]) + 30          # small positions: fp32 angles are exact enough
    tw = {k: torch.tensor(v) for k, v in w.items()}

    def f(x, a):
        h = F.gelu(F.linear(x, tw["w1_" + a], tw["b1_" + a]), approximate="none")
        return F.linear(h, tw["w2_" + a], tw["b2_" + a])

    k = F.linear(f(torch.tensor(V), "v"), tw["w_k"])
    q = F.linear(f(torch.tensor(T), "t"), tw["w_q"])
    emb = llama.LlamaRotaryEmbedding(LlamaConfig(hidden_size=8, num_attention_heads=1, head_dim=8,
                                                 rope_theta=10000.0))
    cv, sv = emb(torch.zeros(1), torch.tensor(pv)[None])
    ct, st = emb(torch.zeros(1), torch.tensor(pt)[None])
    k_rot, _ = llama.apply_rotary_pos_emb(k[None, None], k[None, None], cv.double(), sv.double())
    q_rot, _ = llama.apply_rotary_pos_emb(q[None, None], q[None, None], ct.double(), st.double())
    eye = torch.eye(V.shape[0], dtype=torch.float64)[None, None]
    attn = F.scaled_dot_product_attention(q_rot, k_rot, eye)[0, 0]     # [M, N]
    want = attn.mean(dim=0).numpy()
    np.testing.assert_allclose(predicted_attention(V, T, pv, pt, w), want, rtol=2e-5)


def test_mlp_is_tokenwise():
    rng = np.random.default_rng(2)
    w = _weights(rng, 6, 5, 4)
    X = rng.standard_normal((7, 6))
    full = mlp(X, w["w1_v"], w["b1_v"], w["w2_v"], w["b2_v"])
    for i in range(7):
        np.testing.assert_allclose(full[i], mlp(X[i:i + 1], w["w1_v"], w["b1_v"], w["w2_v"],
                                                w["b2_v"])[0], rtol=1e-14)


def test_peaked_workload_makes_the_bf16_bar_discriminate():
    """On the default workload (weights N(0, 0.02^2)) p_hat is nearly flat,
    and a 10 % error in the logit scale moves it by less than the 2e-2 bf16
    bar; with weights N(0, 0.03^2) the same error moves it by more, and so
    does dropping the bias of f_V's second layer: the GPU score tests run
    that workload so that such mistakes cannot pass."""
    from workloads import PredictorShape, get_config, make_inputs
    names = ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")

    def rel_moves(std):
        cfg = get_config("tiny", N=576, pred=PredictorShape(weight_std=std))
        x = make_inputs(cfg)
        w = {n: x[n + "_f32"].astype(np.float64) for n in names}
        args = (x["V_f32"][0], x["T_f32"], x["pos_v"][0], x["pos_t"])
        p = predicted_attention(*args, w)
        scaled = dict(w, w_q=1.1 * w["w_q"])        # logits times 1.1
        no_bias = dict(w, b2_v=0.0 * w["b2_v"])     # f_V's second bias dropped
        return (np.max(np.abs(predicted_attention(*args, scaled) / p - 1)),
                np.max(np.abs(predicted_attention(*args, no_bias) / p - 1)), p.max() / p.min())

    flat_scale, _, flat_span = rel_moves(0.02)
    assert flat_scale < 2e-2 and flat_span < 1.5
    peaked_scale, peaked_bias, peaked_span = rel_moves(0.03)
    assert peaked_scale > 2e-2 and peaked_bias > 2e-2 and peaked_span > 10
