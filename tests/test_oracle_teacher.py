"""Pins of the teacher-selection oracle (section "Question Contrastive Teacher
Selection", Eq. (1)-(2), QCTS-n of Table 5) against facts fixed outside it:
the textbook entropy form of the Jensen-Shannon divergence, scipy's
implementation, closed forms, explicit loops over heads and tokens, and
planted layers."""
import math

import numpy as np
import pytest
from scipy.spatial.distance import jensenshannon

import oracle
from workloads import make_attention


def _entropy(x):
    x = np.asarray(x, dtype=np.float64)
    return -sum(v * math.log(v) for v in x if v > 0)


def test_js_two_point_closed_form():
    # p = (1, 0), q = (1/2, 1/2): m = (3/4, 1/4), JS = H(m) - (H(p) + H(q)) / 2 = H(m) - ln 2 / 2
    want = -(0.75 * math.log(0.75) + 0.25 * math.log(0.25)) - 0.5 * math.log(2.0)
    assert oracle.js_divergence([1.0, 0.0], [0.5, 0.5]) == pytest.approx(want, rel=1e-14)


def test_js_disjoint_supports_is_ln2_and_identical_is_zero():
    assert oracle.js_divergence([0.5, 0.5, 0, 0], [0, 0, 0.25, 0.75]) == pytest.approx(math.log(2.0), rel=1e-14)
    p = np.random.default_rng(0).dirichlet(np.ones(50))
    assert oracle.js_divergence(p, p) == 0.0


@pytest.mark.parametrize("seed", range(6))
def test_js_entropy_form_scipy_symmetry_and_bounds(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 300))
    p, q = rng.dirichlet(np.full(n, 0.3)), rng.dirichlet(np.full(n, 0.3))
    p[rng.random(n) < 0.2] = 0.0
    p /= p.sum()
    js = oracle.js_divergence(p, q)
    m = 0.5 * (p + q)
    assert js == pytest.approx(_entropy(m) - 0.5 * (_entropy(p) + _entropy(q)), rel=1e-11, abs=1e-15)
    assert js == pytest.approx(jensenshannon(p, q) ** 2, rel=1e-10, abs=1e-15)
    assert js == pytest.approx(oracle.js_divergence(q, p), rel=1e-13)
    assert 0.0 <= js <= math.log(2.0)


def test_layer_distributions_against_loops():
    rng = np.random.default_rng(3)
    L, H, M, N = 3, 2, 4, 5
    A = rng.random((L, H, M, N))
    p = oracle.layer_distributions(A)
    for l in range(L):
        a = [sum(A[l, h, m, n] for h in range(H) for m in range(M)) / (H * M) for n in range(N)]
        s = sum(a)
        for n in range(N):
            assert p[l, n] == pytest.approx(a[n] / s, rel=1e-13)


def test_layer_distributions_hand_example_and_conventions():
    # one layer, two heads, one question token, three visual tokens
    A = np.array([[[[0.1, 0.2, 0.1]], [[0.3, 0.2, 0.1]]]])
    np.testing.assert_allclose(oracle.layer_distributions(A), [[0.4 / 1.0, 0.4 / 1.0, 0.2 / 1.0]], rtol=1e-14)
    # a layer with no attention on the visual tokens: uniform
    np.testing.assert_array_equal(oracle.layer_distributions(np.zeros((1, 2, 2, 4))), np.full((1, 4), 0.25))
    # scaling a layer, or permuting heads and question tokens, changes nothing
    A = np.random.default_rng(4).random((2, 3, 5, 7))
    B = A.copy()
    B[1] *= 7.5
    B = B[:, ::-1, np.random.default_rng(5).permutation(5)]
    np.testing.assert_allclose(oracle.layer_distributions(B), oracle.layer_distributions(A), rtol=1e-13)


def test_selection_finds_planted_layer_and_ranks():
    rng = np.random.default_rng(6)
    L, H, M, N = 6, 2, 3, 40
    A_ref = rng.random((L, H, 2, N))
    A = np.concatenate([A_ref, A_ref], axis=2)   # the same distribution as the reference in every layer
    focus = np.zeros(N)
    focus[:4] = 1.0
    for l, w in ((4, 5.0), (1, 2.0), (2, 0.5)):
        A[l] = A[l] + w * focus                              # the question moves mass onto 4 tokens
    r = oracle.teacher_selection(A, A_ref, n_top=3)
    assert r.js[0] == pytest.approx(0.0, abs=1e-15) and r.js[5] == pytest.approx(0.0, abs=1e-15)
    assert list(r.layers) == [4, 1, 2]
    np.testing.assert_allclose(r.teacher, (r.p[4] + r.p[1] + r.p[2]) / 3, rtol=1e-14)
    one = oracle.teacher_selection(A, A_ref, n_top=1)
    np.testing.assert_array_equal(one.teacher, r.p[4])
    every = oracle.teacher_selection(A, A_ref, n_top=L)
    np.testing.assert_allclose(every.teacher, r.p.mean(axis=0), rtol=1e-14)
    assert sorted(every.layers) == list(range(L))


def test_selection_ties_go_to_the_lower_layer():
    A = np.ones((4, 1, 2, 8))
    r = oracle.teacher_selection(A, A, n_top=4)
    assert list(r.layers) == [0, 1, 2, 3]
    assert r.js.max() == 0.0


def test_synthetic_attention_recipe():
    Af, As = make_attention(8, 2, 3, 64, dtype="bf16")
    assert As.dtype == np.uint16 and Af.shape == (8, 2, 3, 64)
    np.testing.assert_allclose(Af.sum(axis=3), 0.5, rtol=1e-2)
    Rf, _ = make_attention(8, 2, 3, 64, dtype="bf16", reference=True)
    r = oracle.teacher_selection(Af, Rf, n_top=2)
    assert 1 <= r.layers[0] <= 6      # the question field peaks in the middle layers
