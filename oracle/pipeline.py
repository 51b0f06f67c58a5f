"""Oracle for the whole pruning stage -- test infrastructure.

Score (Eq. (3)), select (top-K0, basis, Eq. (4)), restore the original order
and gather the kept rows with their positional indices (section
"Inference-Time Token Pruning").
"""
from dataclasses import dataclass

import numpy as np

from .predictor import predicted_attention
from .select import greedy_select


@dataclass
class PruneResult:
    p_hat: np.ndarray      # [B, N] float64
    idx: np.ndarray        # [B, K] ascending original indices
    order: np.ndarray      # [B, K] selection order
    V_out: np.ndarray      # [B, K, D] kept rows (same dtype as the V given)
    pos_out: np.ndarray    # [B, K] positional indices of the kept rows


def prune(V, T, t_off, pos_v, pos_t, w: dict, K: int, K0: int, tau: float = 1e-2,
          theta: float = 10000.0) -> PruneResult:
    V = np.asarray(V)
    B, N, D = V.shape
    p = np.empty((B, N))
    idx = np.empty((B, K), np.int64)
    order = np.empty((B, K), np.int64)
    for b in range(B):
        lo, hi = int(t_off[b]), int(t_off[b + 1])
        p[b] = predicted_attention(V[b], T[lo:hi], pos_v[b], pos_t[lo:hi], w, theta)
        r = greedy_select(p[b], V[b], K, K0, tau)
        idx[b], order[b] = r.idx, r.order
    V_out = np.take_along_axis(V, idx[:, :, None], axis=1)
    pos_out = np.take_along_axis(np.asarray(pos_v), idx, axis=1)
    return PruneResult(p, idx, order, V_out, pos_out)


def assemble(V_out, pos_out, T, pos_t, t_off):
    """The language model's layer-0 input after pruning (section
    "Inference-Time Token Pruning": the kept tokens, in their original order
    with their positional indices, are combined with the question tokens):
    per image its K kept rows, then its question rows, packed in image order."""
    V_out, pos_out = np.asarray(V_out), np.asarray(pos_out)
    T, pos_t = np.asarray(T), np.asarray(pos_t)
    rows, pos = [], []
    for b in range(V_out.shape[0]):
        lo, hi = int(t_off[b]), int(t_off[b + 1])
        rows += [V_out[b], T[lo:hi]]
        pos += [pos_out[b], pos_t[lo:hi]]
    return np.concatenate(rows, axis=0), np.concatenate(pos)
