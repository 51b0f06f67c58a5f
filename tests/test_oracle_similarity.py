"""Pins of the similarity oracle: the defining properties of a cosine matrix
and torch's own pairwise cosine similarity."""
import numpy as np
import pytest

from oracle import cosine_entries, cosine_similarity, row_norms


def _V(seed=0, N=30, D=17):
    return np.random.default_rng(seed).standard_normal((N, D))


def test_cosine_properties():
    S = cosine_similarity(_V())
    np.testing.assert_allclose(S, S.T, atol=0)
    np.testing.assert_allclose(np.diag(S), 1.0, atol=1e-15)
    assert np.all(np.abs(S) <= 1 + 1e-15)


def test_matches_torch_cosine_similarity():
    torch = pytest.importorskip("torch")
    V = _V(1)
    t = torch.tensor(V)
    want = torch.nn.functional.cosine_similarity(t[:, None, :], t[None, :, :], dim=-1, eps=0.0)
    np.testing.assert_allclose(cosine_similarity(V), want.numpy(), atol=1e-14)


def test_norms_textbook():
    np.testing.assert_allclose(row_norms(np.array([[3.0, 4.0], [0.0, 0.0]])), [5.0, 0.0])


def test_zero_row_convention_and_entries():
    V = _V(2)
    V[4] = 0.0
    S = cosine_similarity(V)
    assert np.all(S[4] == 0) and np.all(S[:, 4] == 0)
    rng = np.random.default_rng(3)
    rows, cols = rng.integers(0, 30, 50), rng.integers(0, 30, 50)
    np.testing.assert_allclose(cosine_entries(V, rows, cols), S[rows, cols], atol=1e-15)
