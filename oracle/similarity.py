"""Oracle for the visual-token norms and cosine similarity -- test infrastructure.

The diversity term of Eq. (4) (section "Inference-Time Token Pruning") uses
the raw visual embeddings v_i.  Their norms n_i = ||v_i|| and the cosine
similarity S_ij = <v_i, v_j> / (n_i n_j) are the pairwise quantities a
Gram-based evaluation of that residual consumes.  A zero row has norm 0 and,
by the convention used throughout, a zero row and column in S.
"""
import numpy as np


def row_norms(V) -> np.ndarray:
    V = np.asarray(V, np.float64)
    return np.sqrt((V * V).sum(axis=-1))


def _inv(n):
    out = np.zeros_like(n)
    nz = n > 0
    out[nz] = 1.0 / n[nz]
    return out


def cosine_similarity(V) -> np.ndarray:
    """S [N, N] of one image V [N, D], float64."""
    V = np.asarray(V, np.float64)
    ninv = _inv(row_norms(V))
    return (V @ V.T) * ninv[:, None] * ninv[None, :]


def cosine_entries(V, rows, cols) -> np.ndarray:
    """S[rows[k], cols[k]] one by one, for spot checks at large N."""
    V = np.asarray(V, np.float64)
    rows = np.asarray(rows)
    cols = np.asarray(cols)
    a, b = V[rows], V[cols]
    na, nb = row_norms(a), row_norms(b)
    dots = (a * b).sum(axis=1)
    return dots * _inv(na) * _inv(nb)
