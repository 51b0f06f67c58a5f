"""Pins of the training-step oracle (the KL objective of section
"Cross-Modal Attention Distillation" and its gradient) to things other than
itself: textbook values of GELU' and of the divergence, scipy's relative
entropy, central finite differences of the loss, torch autograd of an
independently written forward pass, and the divergence's minimum (a teacher
equal to p_hat gives zero loss and zero gradient).  Planted mistakes in the
chain rule must fail the finite-difference check."""
import math

import numpy as np
import pytest

import oracle.train as tr
from oracle import predicted_attention_batch

PHI_1, PDF_1 = 0.8413447460685429, 0.24197072451914337   # Phi(1), phi(1)


def test_gelu_grad_textbook_values():
    got = tr.gelu_erf_grad(np.array([0.0, 1.0, -1.0]))
    np.testing.assert_allclose(got, [0.5, PHI_1 + PDF_1, (1 - PHI_1) - PDF_1], rtol=0, atol=1e-15)
    x = np.linspace(-4, 4, 33)
    h = 1e-6
    fd = (tr.gelu_erf(x + h) - tr.gelu_erf(x - h)) / (2 * h)
    np.testing.assert_allclose(tr.gelu_erf_grad(x), fd, atol=1e-9)


def test_kl_hand_values_and_scipy():
    from scipy.special import rel_entr
    assert tr.kl_divergence([0.5, 0.5, 0.0], [0.25, 0.5, 0.25]) == pytest.approx(0.5 * math.log(2.0), abs=1e-16)
    p = np.array([0.1, 0.2, 0.7])
    assert tr.kl_divergence(p, p) == 0.0
    q = np.array([0.3, 0.3, 0.4])
    assert tr.kl_divergence(p, q) == pytest.approx(float(np.sum(rel_entr(p, q))), rel=1e-15)


def _case(seed=0, B=2, N=7, Ms=(3, 2), D=6, H=5, dp=4, scale=0.5):
    rng = np.random.default_rng(seed)
    w = {k: scale * rng.standard_normal(s) for k, s in
         [("w1_v", (H, D)), ("b1_v", (H,)), ("w2_v", (H, H)), ("b2_v", (H,)), ("w_k", (dp, H)),
          ("w1_t", (H, D)), ("b1_t", (H,)), ("w2_t", (H, H)), ("b2_t", (H,)), ("w_q", (dp, H))]}
    V = rng.standard_normal((B, N, D))
    t_off = np.concatenate([[0], np.cumsum(Ms)])
    T = rng.standard_normal((t_off[-1], D))
    pos_v = np.stack([np.arange(N) + 3 * b for b in range(B)])
    pos_t = N + rng.integers(0, 6, size=t_off[-1])
    p_star = rng.dirichlet(np.ones(N), size=B)
    p_star[0, 2] = 0.0                      # a zero teacher entry (0 log 0 = 0)
    p_star[0] /= p_star[0].sum()
    return V, T, t_off, pos_v, pos_t, w, p_star


def _fd_check(step):
    """Central differences of the batch loss against `step`'s gradient, entry by entry."""
    V, T, t_off, pos_v, pos_t, w, p_star = _case()
    r = step(V, T, t_off, pos_v, pos_t, w, p_star)
    h = 1e-5
    for name in tr.PARAMS:
        fd = np.empty_like(w[name])
        for i in np.ndindex(w[name].shape):
            wp = {k: v.copy() for k, v in w.items()}
            wm = {k: v.copy() for k, v in w.items()}
            wp[name][i] += h
            wm[name][i] -= h
            fd[i] = (tr.train_step(V, T, t_off, pos_v, pos_t, wp, p_star).loss -
                     tr.train_step(V, T, t_off, pos_v, pos_t, wm, p_star).loss) / (2 * h)
        np.testing.assert_allclose(r.grads[name], fd, rtol=1e-6, atol=1e-9, err_msg=name)


def test_gradients_match_central_differences():
    _fd_check(tr.train_step)


def test_loss_is_the_mean_of_image_divergences():
    V, T, t_off, pos_v, pos_t, w, p_star = _case()
    r = tr.train_step(V, T, t_off, pos_v, pos_t, w, p_star)
    p = predicted_attention_batch(V, T, t_off, pos_v, pos_t, w)
    np.testing.assert_allclose(r.p_hat, p, rtol=1e-14)
    want = [float(np.sum(np.where(p_star[b] > 0, p_star[b] * np.log(np.where(p_star[b] > 0, p_star[b], 1) / p[b]), 0)))
            for b in range(2)]
    np.testing.assert_allclose(r.image_loss, want, rtol=1e-13)
    assert r.loss == pytest.approx(np.mean(want), rel=1e-14)


def test_teacher_equal_to_prediction_is_a_minimum():
    V, T, t_off, pos_v, pos_t, w, _ = _case(seed=4)
    p = predicted_attention_batch(V, T, t_off, pos_v, pos_t, w)
    r = tr.train_step(V, T, t_off, pos_v, pos_t, w, p)
    assert abs(r.loss) < 1e-15
    for name in tr.PARAMS:
        assert np.max(np.abs(r.grads[name])) < 1e-13, name


def test_gradients_match_torch_autograd():
    """The same forward pass written with torch modules (Linear, exact GELU,
    the LLaMA rotary embedding of transformers, softmax, mean) and torch's
    KL divergence, differentiated by autograd in float64."""
    torch = pytest.importorskip("torch")
    llama = pytest.importorskip("transformers.models.llama.modeling_llama")
    from transformers import LlamaConfig
    F = torch.nn.functional
    V, T, t_off, pos_v, pos_t, w, p_star = _case(seed=9, N=11, Ms=(4, 1), D=8, H=6, dp=8)
    tw = {k: torch.tensor(v, requires_grad=True) for k, v in w.items()}
    emb = llama.LlamaRotaryEmbedding(LlamaConfig(hidden_size=8, num_attention_heads=1, head_dim=8,
                                                 rope_theta=10000.0))

    def rot(x, pos):
        # transformers holds its inverse frequencies in float32; the same
        # frequencies (base^(-2i/d)) in float64, then its rotate-half rotation
        inv = 1.0 / (10000.0 ** (torch.arange(0, 8, 2, dtype=torch.float64) / 8))
        np.testing.assert_allclose(inv.numpy(), emb.inv_freq.double().numpy(), rtol=1e-7)
        ang = torch.tensor(pos, dtype=torch.float64)[:, None] * inv[None, :]
        c, s = torch.cat([ang.cos()] * 2, dim=1)[None], torch.cat([ang.sin()] * 2, dim=1)[None]
        out, _ = llama.apply_rotary_pos_emb(x[None, None], x[None, None], c, s)
        return out[0, 0]

    def f(x, a):
        h = F.gelu(F.linear(x, tw["w1_" + a], tw["b1_" + a]), approximate="none")
        return F.linear(h, tw["w2_" + a], tw["b2_" + a])

    total = 0.0
    for b in range(2):
        lo, hi = int(t_off[b]), int(t_off[b + 1])
        k = rot(F.linear(f(torch.tensor(V[b]), "v"), tw["w_k"]), pos_v[b])
        q = rot(F.linear(f(torch.tensor(T[lo:hi]), "t"), tw["w_q"]), pos_t[lo:hi])
        p_hat = torch.softmax(q @ k.T / math.sqrt(8), dim=1).mean(dim=0)
        total = total + F.kl_div(p_hat.log(), torch.tensor(p_star[b]), reduction="sum") / 2
    total.backward()
    r = tr.train_step(V, T, t_off, pos_v, pos_t, w, p_star)
    assert r.loss == pytest.approx(total.item(), rel=1e-12)
    for name in tr.PARAMS:
        np.testing.assert_allclose(r.grads[name], tw[name].grad.numpy(), rtol=1e-9, atol=1e-13, err_msg=name)


def _planted(monkeypatch, what):
    if what == "gelu_grad_phi_only":       # the x phi(x) term dropped
        monkeypatch.setattr(tr, "gelu_erf_grad", lambda x: 0.5 * (1.0 + tr.erf(np.asarray(x) / np.sqrt(2.0))))
    elif what == "rope_forward_angle":     # RoPE's transpose taken as the rotation itself
        real = tr.rope
        monkeypatch.setattr(tr, "rope", lambda x, pos, theta: real(x, np.abs(np.asarray(pos, np.float64)), theta))
    elif what == "missing_sqrt_d":         # the logits' 1/sqrt(d) left out of the backward
        real = tr._branch_backward

        def wrong(X, a, h, u, w2, wp, dz, g, s):
            return real(X, a, h, u, w2, wp, np.sqrt(dz.shape[1]) * dz, g, s)
        monkeypatch.setattr(tr, "_branch_backward", wrong)


@pytest.mark.parametrize("what", ["gelu_grad_phi_only", "rope_forward_angle", "missing_sqrt_d"])
def test_finite_differences_reject_planted_mistakes(monkeypatch, what):
    V, T, t_off, pos_v, pos_t, w, p_star = _case()
    good = tr.train_step(V, T, t_off, pos_v, pos_t, w, p_star)
    _planted(monkeypatch, what)
    bad = tr.train_step(V, T, t_off, pos_v, pos_t, w, p_star)
    monkeypatch.undo()
    assert any(np.max(np.abs(bad.grads[k] - good.grads[k])) > 1e-6 * (1 + np.max(np.abs(good.grads[k])))
               for k in tr.PARAMS)
    with pytest.raises(AssertionError):
        _fd_check(lambda *a: bad)
