"""Oracle for the language model's first layer over the pruned input --
test infrastructure.

Paper, section "Inference-Time Token Pruning": after pruning, the K kept
visual tokens (in their original order, with their original positional
indices) and the question tokens form the language model's input, and the
model processes only those K + M tokens; this is where the method's prefill
and end-to-end speedups come from (Table 7).  The language models evaluated
(LLaVA-1.5 / LLaVA-NeXT on Vicuna-7B) use the LLaMA decoder layer:

    h   = RMSNorm(x) * g_attn
    q, k, v = h W_q^T, h W_k^T, h W_v^T, split into heads of width d_h
    q, k  rotated per head by RoPE at each token's positional index
    o   = softmax(q k^T / sqrt(d_h) + causal mask) v   (per sequence, per head)
    x1  = x + o W_o^T
    y   = x1 + (SiLU(h2 W_g^T) * (h2 W_u^T)) W_d^T,   h2 = RMSNorm(x1) * g_ffn

Readings (each also listed in the design notes): the layer is LLaMA's
(Vicuna-7B: d = 4096, 32 heads of 128, SwiGLU width 11008, RMSNorm
eps = 1e-6 -- the paper names the models, not their layers); RoPE pairs
(i, i + d_h/2) within each head with frequencies theta^(-2i/d_h); the causal
mask follows the row order of each sequence (image b's kept rows, then its
question rows), while RoPE uses the positional indices the rows carry.

Everything is float64; matrix products and the exponential are library
primitives; nothing is fused.
"""
import numpy as np

from .predictor import rope

PARAMS = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g, row by row."""
    x = np.asarray(x, np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(g, np.float64)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """One head of one sequence: softmax(q k^T / sqrt(d_h)) v with row i
    attending to rows j <= i."""
    S, dh = q.shape
    logits = q @ k.T / np.sqrt(dh)
    logits = np.where(np.tril(np.ones((S, S), bool)), logits, -np.inf)
    e = np.exp(logits - logits.max(axis=1, keepdims=True))
    return (e / e.sum(axis=1, keepdims=True)) @ v


def decoder_layer(X, pos, seq_off, p: dict, n_heads: int, theta: float = 10000.0, eps: float = 1e-6):
    """Y [R, d] for the packed sequences X [R, d]: sequence b holds rows
    seq_off[b] .. seq_off[b+1]-1, row r at positional index pos[r].
    ``p``: attn_norm [d], w_qkv [3d, d] (W_q, W_k, W_v stacked), w_o [d, d],
    ffn_norm [d], w_gate_up [2 ff, d] (W_g then W_u), w_down [d, ff]."""
    X = np.asarray(X, np.float64)
    g = {k: np.asarray(v, np.float64) for k, v in p.items()}
    R, d = X.shape
    dh = d // n_heads
    ff = g["w_down"].shape[1]
    h = rms_norm(X, g["attn_norm"], eps)
    qkv = h @ g["w_qkv"].T
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    o = np.zeros((R, d))
    for b in range(len(seq_off) - 1):
        lo, hi = int(seq_off[b]), int(seq_off[b + 1])
        for hd in range(n_heads):
            cols = slice(hd * dh, (hd + 1) * dh)
            qh = rope(q[lo:hi, cols], pos[lo:hi], theta)
            kh = rope(k[lo:hi, cols], pos[lo:hi], theta)
            o[lo:hi, cols] = causal_attention(qh, kh, v[lo:hi, cols])
    x1 = X + o @ g["w_o"].T
    h2 = rms_norm(x1, g["ffn_norm"], eps)
    gu = h2 @ g["w_gate_up"].T
    return x1 + (silu(gu[:, :ff]) * gu[:, ff:]) @ g["w_down"].T
