"""Oracle for the predicted attention of Eq. (3) -- test infrastructure.

Paper, section "Cross-Modal Attention Distillation": the predictor maps the
question tokens t_m and the visual tokens v_n through two modality-specific
MLPs f_T and f_V, projects them with W_Q (text) and W_K (visual), applies RoPE
to the projected queries and keys, and computes

    p_hat_n = (1/M) sum_m softmax_n( <W_Q f_T(t_m), W_K f_V(v_n)> / sqrt(d) ),

d being the projection width.  Value and output projections do not exist.

Readings of what the paper leaves open (each also listed in the design notes):
* f_T, f_V: Linear(D -> D_h) + bias, GELU (erf form), Linear(D_h -> D_h) + bias.
* W_Q, W_K: Linear(D_h -> d) without bias; one head (Eq. (3) has no head index).
* RoPE: rotate-half pairing (i, i + d/2), frequency theta^(-2i/d), positions
  given explicitly per token.
* The softmax runs over the N visual tokens only (so p_hat sums to one), then
  the rows are averaged over the M question tokens (softmax first, then mean:
  the active form of Eq. (3)).

Everything is float64.  Matrix products and erf are library primitives; no
blocking or fusion is done.
"""
import numpy as np
from scipy.special import erf


def gelu_erf(x: np.ndarray) -> np.ndarray:
    """GELU, exact erf form: x * Phi(x)."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def mlp(x: np.ndarray, w1, b1, w2, b2) -> np.ndarray:
    """Modality MLP f(x) = W2 GELU(W1 x + b1) + b2, applied token-wise.
    Weights use the W[out][in] layout."""
    h = gelu_erf(x @ np.asarray(w1, np.float64).T + np.asarray(b1, np.float64))
    return h @ np.asarray(w2, np.float64).T + np.asarray(b2, np.float64)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary position embedding of rows x [n, d] at integer positions pos [n].

    Pair i (i < d/2) is (x[:, i], x[:, i + d/2]) and rotates by the angle
    pos * theta^(-2i/d):  (a, b) -> (a cos - b sin, b cos + a sin).
    """
    n, d = x.shape
    if d % 2:
        raise ValueError("RoPE needs an even width")
    half = d // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / d)
    ang = np.asarray(pos, np.float64)[:, None] * inv_freq[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[:, :half], x[:, half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=1)


def predicted_attention(V, T, pos_v, pos_t, w: dict, theta: float = 10000.0) -> np.ndarray:
    """p_hat [N] of one image, Eq. (3).

    V [N, D] visual tokens, T [M, D] question tokens, pos_v [N], pos_t [M];
    ``w`` maps w1_v, b1_v, w2_v, b2_v, w_k, w1_t, b1_t, w2_t, b2_t, w_q to arrays.
    """
    V = np.asarray(V, np.float64)
    T = np.asarray(T, np.float64)
    g = {k: np.asarray(v, np.float64) for k, v in w.items()}
    keys = rope(mlp(V, g["w1_v"], g["b1_v"], g["w2_v"], g["b2_v"]) @ g["w_k"].T, pos_v, theta)
    queries = rope(mlp(T, g["w1_t"], g["b1_t"], g["w2_t"], g["b2_t"]) @ g["w_q"].T, pos_t, theta)
    d = keys.shape[1]
    logits = queries @ keys.T / np.sqrt(d)                     # [M, N]
    logits = logits - logits.max(axis=1, keepdims=True)
    e = np.exp(logits)
    attn = e / e.sum(axis=1, keepdims=True)                    # softmax over n
    return attn.mean(axis=0)                                   # mean over m


def predicted_attention_batch(V, T, t_off, pos_v, pos_t, w: dict, theta: float = 10000.0):
    """p_hat [B, N] for a batch: V [B, N, D], T [sum M, D] with offsets t_off."""
    B = V.shape[0]
    out = np.empty((B, V.shape[1]), np.float64)
    for b in range(B):
        lo, hi = int(t_off[b]), int(t_off[b + 1])
        out[b] = predicted_attention(V[b], T[lo:hi], pos_v[b], pos_t[lo:hi], w, theta)
    return out
