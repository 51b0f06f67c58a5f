"""Pins of the batched oracle functions: predicted_attention_batch (Eq. (3)
per image, with ragged questions) and pipeline.prune (score, select, restore
the original order, gather; section "Inference-Time Token Pruning").

Both are pinned by hand-worked values, not by calls of the functions they
are built from:
* the batch of Eq. (3) uses the two-wide identity predictor of the worked
  example in test_oracle_predictor: every p_hat follows from the normal-CDF
  table, and RoPE at integer positions turns a logit by the cosine of the
  position difference;
* prune uses W_Q = 0 (p_hat uniform, 1/N exactly) and mutually orthogonal
  rows of distinct norms, so the greedy order is the order of the norms and
  every index, position and row is written out.
Each pin is also run against a copy of the function with a planted mistake
(a shifted question slice, another image's positions, a gather by selection
order instead of ascending index) and must reject it."""
import math

import numpy as np
import pytest

import oracle
from oracle import predicted_attention
from oracle.select import greedy_select

PHI_1 = 0.8413447460685429   # Phi(1)
PHI_2 = 0.9772498680518208   # Phi(2)

I2, Z2 = np.eye(2), np.zeros(2)
IDENTITY = {"w1_v": I2, "b1_v": Z2, "w2_v": I2, "b2_v": Z2, "w_k": I2,
            "w1_t": I2, "b1_t": Z2, "w2_t": I2, "b2_t": Z2, "w_q": I2}


def _softmax(x):
    e = [math.exp(v) for v in x]
    return [v / sum(e) for v in e]


def _batch_case():
    """Four images of the same three visual rows (0,0), (1,0), (2,0) -- keys
    0, Phi(1), 2 Phi(2) on the first axis -- with ragged questions:
      image 0: questions (1,0), (0,0) at position 0  (the worked example)
      image 1: question (0,0)                        (all logits 0: uniform)
      image 2: question (1,0), visual rows reversed  (p reversed)
      image 3: question (1,0) at position 3, keys at 0 (logits times cos 3)
    """
    rows = np.array([[0.0, 0.0], [1.0, 0.0], [2.0, 0.0]])
    V = np.stack([rows, rows, rows[::-1], rows])
    T = np.array([[1.0, 0.0], [0.0, 0.0], [0.0, 0.0], [1.0, 0.0], [1.0, 0.0]])
    t_off = np.array([0, 2, 3, 4, 5])
    pos_v = np.zeros((4, 3), np.int64)
    pos_t = np.array([0, 0, 0, 0, 3])
    keys = [0.0, PHI_1, 2 * PHI_2]
    q = PHI_1
    one = _softmax([q * k / math.sqrt(2) for k in keys])
    want = np.array([
        [0.5 * (one[i] + 1.0 / 3.0) for i in range(3)],
        [1.0 / 3.0] * 3,
        one[::-1],
        _softmax([q * k * math.cos(3.0) / math.sqrt(2) for k in keys]),
    ])
    return V, T, t_off, pos_v, pos_t, want


def _check_batch(fn):
    V, T, t_off, pos_v, pos_t, want = _batch_case()
    got = fn(V, T, t_off, pos_v, pos_t, IDENTITY)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=0)


def test_batch_hand_worked_ragged_questions():
    _check_batch(oracle.predicted_attention_batch)


def _batch_shifted_slice(V, T, t_off, pos_v, pos_t, w):
    """Planted mistake: each image reads the question rows one place late."""
    out = np.empty((V.shape[0], V.shape[1]))
    for b in range(V.shape[0]):
        lo, hi = int(t_off[b]) + 1, int(t_off[b + 1]) + 1
        out[b] = predicted_attention(V[b], T[lo:hi], pos_v[b], pos_t[lo:hi], w)
    return out


def _batch_first_question_only(V, T, t_off, pos_v, pos_t, w):
    """Planted mistake: every image scored against image 0's question."""
    lo, hi = int(t_off[0]), int(t_off[1])
    return np.stack([predicted_attention(V[b], T[lo:hi], pos_v[b], pos_t[lo:hi], w) for b in range(V.shape[0])])


def _batch_positions_of_image0(V, T, t_off, pos_v, pos_t, w):
    """Planted mistake: the question positions of the first question token
    used for every question token."""
    out = np.empty((V.shape[0], V.shape[1]))
    for b in range(V.shape[0]):
        lo, hi = int(t_off[b]), int(t_off[b + 1])
        out[b] = predicted_attention(V[b], T[lo:hi], pos_v[b], np.full(hi - lo, pos_t[0]), w)
    return out


@pytest.mark.filterwarnings("ignore::RuntimeWarning")  # the shifted slice leaves the last image empty
@pytest.mark.parametrize("planted", [_batch_shifted_slice, _batch_first_question_only, _batch_positions_of_image0])
def test_batch_pin_rejects_planted_mistakes(planted):
    with pytest.raises(AssertionError):
        _check_batch(planted)


def test_batch_permuting_images_permutes_rows():
    rng = np.random.default_rng(7)
    B, N, D, H, dp = 3, 9, 6, 5, 4
    w = {k: 0.4 * rng.standard_normal(s) for k, s in
         [("w1_v", (H, D)), ("b1_v", (H,)), ("w2_v", (H, H)), ("b2_v", (H,)), ("w_k", (dp, H)),
          ("w1_t", (H, D)), ("b1_t", (H,)), ("w2_t", (H, H)), ("b2_t", (H,)), ("w_q", (dp, H))]}
    V = rng.standard_normal((B, N, D))
    lens = [2, 5, 1]
    t_off = np.concatenate([[0], np.cumsum(lens)])
    T = rng.standard_normal((t_off[-1], D))
    pos_v = np.stack([np.arange(N) + 13 * b for b in range(B)])
    pos_t = rng.integers(0, 50, size=t_off[-1])
    p = oracle.predicted_attention_batch(V, T, t_off, pos_v, pos_t, w)
    perm = [2, 0, 1]
    T2 = np.concatenate([T[t_off[b]:t_off[b + 1]] for b in perm])
    pt2 = np.concatenate([pos_t[t_off[b]:t_off[b + 1]] for b in perm])
    off2 = np.concatenate([[0], np.cumsum([lens[b] for b in perm])])
    p2 = oracle.predicted_attention_batch(V[perm], T2, off2, pos_v[perm], pt2, w)
    np.testing.assert_array_equal(p2, p[perm])
    assert np.all(np.abs(p[0] - p[1]) > 0)  # the images' rows differ, so a mix-up would show


# ---------------------------------------------------------------- prune

def _prune_case():
    """Two images of five mutually orthogonal rows (distinct axes of R^8)
    with distinct norms, W_Q = 0 so p_hat = 1/5 exactly.  Eq. (4)'s score is
    then norm / 5 for every token not yet kept (orthogonal rows keep their
    whole norm as residual), so the greedy order is the order of the norms.
      image 0: norms 1, 3, 2, 5, 4   -> K0 = 0 order 3, 4, 1
      image 1: norms 4, 1, 5, 2, 3   -> K0 = 0 order 2, 0, 4
    With K0 = 1 the top-K0 of a flat p_hat is token 0 (ties to the lower
    index), then the largest norms follow:
      image 0: order 0, 3, 4;  image 1: order 0, 2, 4."""
    D = 8
    norms = [[1.0, 3.0, 2.0, 5.0, 4.0], [4.0, 1.0, 5.0, 2.0, 3.0]]
    axes = [[6, 1, 4, 0, 3], [2, 7, 5, 1, 0]]
    V = np.zeros((2, 5, D), np.float32)
    for b in range(2):
        for i in range(5):
            V[b, i, axes[b][i]] = norms[b][i]
    rng = np.random.default_rng(11)
    T = rng.standard_normal((3, D))
    t_off = np.array([0, 1, 3])
    pos_v = np.array([[10, 11, 12, 13, 14], [7, 3, 9, 1, 5]])
    pos_t = np.array([5, 5, 6])
    H, dp = 4, 2
    w = {"w1_v": rng.standard_normal((H, D)), "b1_v": rng.standard_normal(H),
         "w2_v": rng.standard_normal((H, H)), "b2_v": rng.standard_normal(H),
         "w_k": rng.standard_normal((dp, H)),
         "w1_t": rng.standard_normal((H, D)), "b1_t": rng.standard_normal(H),
         "w2_t": rng.standard_normal((H, H)), "b2_t": rng.standard_normal(H),
         "w_q": np.zeros((dp, H))}
    return V, T, t_off, pos_v, pos_t, w


PRUNE_WANT = {
    0: dict(order=[[3, 4, 1], [2, 0, 4]], idx=[[1, 3, 4], [0, 2, 4]], pos=[[11, 13, 14], [7, 9, 5]]),
    1: dict(order=[[0, 3, 4], [0, 2, 4]], idx=[[0, 3, 4], [0, 2, 4]], pos=[[10, 13, 14], [7, 9, 5]]),
}


def _check_prune(fn, K0):
    V, T, t_off, pos_v, pos_t, w = _prune_case()
    r = fn(V, T, t_off, pos_v, pos_t, w, 3, K0, 1e-2)
    want = PRUNE_WANT[K0]
    np.testing.assert_array_equal(r.p_hat, np.full((2, 5), 0.2))
    np.testing.assert_array_equal(r.order, want["order"])
    np.testing.assert_array_equal(r.idx, want["idx"])
    np.testing.assert_array_equal(r.pos_out, want["pos"])
    assert r.V_out.dtype == V.dtype
    for b in range(2):
        for k, i in enumerate(want["idx"][b]):
            assert r.V_out[b, k].tobytes() == V[b, i].tobytes()


@pytest.mark.parametrize("K0", [0, 1])
def test_prune_hand_worked_two_images(K0):
    _check_prune(oracle.prune, K0)


def _prune_gather_by_order(V, T, t_off, pos_v, pos_t, w, K, K0, tau):
    """Planted mistake: rows and positions gathered in selection order."""
    r = oracle.prune(V, T, t_off, pos_v, pos_t, w, K, K0, tau)
    r.V_out = np.take_along_axis(V, r.order[:, :, None], axis=1)
    r.pos_out = np.take_along_axis(pos_v, r.order, axis=1)
    r.idx = r.order
    return r


def _prune_positions_by_rank(V, T, t_off, pos_v, pos_t, w, K, K0, tau):
    """Planted mistake: positions renumbered 0..K-1 instead of gathered."""
    r = oracle.prune(V, T, t_off, pos_v, pos_t, w, K, K0, tau)
    r.pos_out = np.tile(np.arange(K), (V.shape[0], 1))
    return r


def _prune_image0_selection(V, T, t_off, pos_v, pos_t, w, K, K0, tau):
    """Planted mistake: every image keeps image 0's selection."""
    r = oracle.prune(V, T, t_off, pos_v, pos_t, w, K, K0, tau)
    r.idx = np.tile(r.idx[:1], (V.shape[0], 1))
    r.order = np.tile(r.order[:1], (V.shape[0], 1))
    r.V_out = np.take_along_axis(V, r.idx[:, :, None], axis=1)
    r.pos_out = np.take_along_axis(pos_v, r.idx, axis=1)
    return r


@pytest.mark.parametrize("planted", [_prune_gather_by_order, _prune_positions_by_rank, _prune_image0_selection])
def test_prune_pin_rejects_planted_mistakes(planted):
    with pytest.raises(AssertionError):
        _check_prune(planted, 0)


def test_prune_scores_each_image_with_its_own_question():
    """prune's p_hat equals the pinned batch function's on a ragged batch
    (different question lengths and positions per image), and its
    selection is greedy_select on that p_hat."""
    rng = np.random.default_rng(3)
    B, N, D, H, dp = 3, 12, 8, 6, 4
    w = {k: 0.5 * rng.standard_normal(s) for k, s in
         [("w1_v", (H, D)), ("b1_v", (H,)), ("w2_v", (H, H)), ("b2_v", (H,)), ("w_k", (dp, H)),
          ("w1_t", (H, D)), ("b1_t", (H,)), ("w2_t", (H, H)), ("b2_t", (H,)), ("w_q", (dp, H))]}
    V = rng.standard_normal((B, N, D))
    t_off = np.array([0, 3, 4, 9])
    T = rng.standard_normal((9, D))
    pos_v = np.stack([np.arange(N) + 5 * b for b in range(B)])
    pos_t = N + rng.integers(0, 9, size=9)
    r = oracle.prune(V, T, t_off, pos_v, pos_t, w, 5, 2)
    p = oracle.predicted_attention_batch(V, T, t_off, pos_v, pos_t, w)
    np.testing.assert_array_equal(r.p_hat, p)
    for b in range(B):
        np.testing.assert_array_equal(r.order[b], greedy_select(p[b], V[b], 5, 2).order)
