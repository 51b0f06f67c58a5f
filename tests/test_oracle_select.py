"""Pins of the selection oracle (Eq. (4)) to things other than itself:
the Top-K special case, LAPACK's QR with column pivoting, brute-force
determinants on tiny inputs, closed forms on orthogonal inputs, and the
invariants the rule implies."""

import numpy as np
import pytest
import scipy.linalg

from oracle import greedy_select, replay_check, restore_order, top_k0


def _data(seed, N, D, p_spread=0.5):
    rng = np.random.default_rng(seed)
    V = rng.standard_normal((N, D))
    p = rng.random(N) * p_spread + 0.5
    return p / p.sum(), V


def test_diversity_off_is_top_k():
    """K0 = K keeps exactly the K largest p_hat (the Top-K baseline row of the
    diversity ablation table)."""
    p, V = _data(0, 50, 16)
    r = greedy_select(p, V, K=12, K0=12)
    want = np.argsort(-p, kind="stable")[:12]
    np.testing.assert_array_equal(r.order, want)
    np.testing.assert_array_equal(r.idx, np.sort(want))


def test_top_k0_ties_prefer_lower_index():
    p = np.array([0.1, 0.3, 0.3, 0.2, 0.3])
    np.testing.assert_array_equal(top_k0(p, 3), [1, 2, 4])


@pytest.mark.parametrize("seed", range(6))
def test_k0_zero_equals_qr_column_pivoting(seed):
    """K0 = 0: scaling column i of V^T by p_i scales its residual by p_i and
    keeps the span, so the picks are the pivots of QR with column pivoting
    (Businger-Golub, LAPACK xGEQP3) of V^T diag(p)."""
    p, V = _data(seed, 40, 64)
    _, _, piv = scipy.linalg.qr(V.T * p[None, :], pivoting=True, mode="economic")
    r = greedy_select(p, V, K=20, K0=0)
    np.testing.assert_array_equal(r.order, piv[:20])


@pytest.mark.parametrize("seed", range(4))
def test_greedy_after_init_equals_qr_pivoting_of_projected_candidates(seed):
    """K0 > 0: after projecting span(R0) out of the candidates (basis from
    numpy's Householder QR, not the oracle's Gram-Schmidt), the greedy picks
    are the column-pivoting order of the projected, p-scaled candidates."""
    p, V = _data(seed + 10, 60, 80)
    K, K0 = 25, 9
    R0 = np.argsort(-p, kind="stable")[:K0]
    Q, _ = np.linalg.qr(V[R0].T)
    cand = np.setdiff1d(np.arange(60), R0)
    X = V[cand].T - Q @ (Q.T @ V[cand].T)
    _, _, piv = scipy.linalg.qr(X * p[cand][None, :], pivoting=True, mode="economic")
    r = greedy_select(p, V, K=K, K0=K0)
    np.testing.assert_array_equal(r.order[:K0], R0)
    np.testing.assert_array_equal(r.order[K0:], cand[piv[:K - K0]])


@pytest.mark.parametrize("seed", range(8))
def test_brute_force_determinants_tiny(seed):
    """Each greedy pick maximises det(L[R + i]) with L = diag(p) V V^T diag(p)
    (Schur complement: det(L[R+i]) / det(L[R]) = p_i^2 ||r_i||^2); checked
    with explicit determinants for N <= 10."""
    rng = np.random.default_rng(seed)
    N, D = rng.integers(4, 11), 12
    p, V = _data(seed + 100, N, D)
    K0 = int(rng.integers(0, 3))
    K = int(rng.integers(K0 + 1, N + 1))
    L = (p[:, None] * V) @ (p[:, None] * V).T
    r = greedy_select(p, V, K=K, K0=K0)
    R = list(r.order[:K0])
    for t in range(K0, K):
        dets = {i: np.linalg.det(L[np.ix_(R + [i], R + [i])]) for i in range(N) if i not in R}
        best = max(dets, key=lambda i: (dets[i], -i))
        assert r.order[t] == best
        R.append(best)
    if K0 == 0:
        np.testing.assert_allclose(np.linalg.det(L[np.ix_(R, R)]), np.prod(r.gain) ** 2, rtol=1e-9)


def test_brute_force_subsets_for_two_picks():
    """With K0 = 0 and K = 2, the greedy pair is: the token with the largest
    p_i ||v_i||, then the one maximising det of the 2 x 2 kernel."""
    p, V = _data(3, 8, 5)
    L = (p[:, None] * V) @ (p[:, None] * V).T
    first = int(np.argmax(np.diag(L)))
    second = max((i for i in range(8) if i != first),
                 key=lambda i: np.linalg.det(L[np.ix_([first, i], [first, i])]))
    r = greedy_select(p, V, K=2, K0=0)
    assert list(r.order) == [first, second]


def test_orthogonal_rows_reduce_to_ranking_by_p_times_norm():
    rng = np.random.default_rng(4)
    Q, _ = np.linalg.qr(rng.standard_normal((30, 30)))
    norms = rng.random(30) + 0.5
    V = Q * norms[:, None]
    p = rng.random(30); p /= p.sum()
    r = greedy_select(p, V, K=15, K0=5)
    R0 = np.argsort(-p, kind="stable")[:5]
    rest = np.setdiff1d(np.arange(30), R0)
    want = rest[np.argsort(-(p[rest] * norms[rest]), kind="stable")[:10]]
    np.testing.assert_array_equal(r.order[5:], want)
    np.testing.assert_allclose(r.gain[5:], (p * norms)[want], rtol=1e-12)


def test_gains_non_increasing_and_indices_valid():
    p, V = _data(5, 200, 48)
    r = greedy_select(p, V, K=60, K0=20)
    g = r.gain[20:]
    assert np.all(np.diff(g) <= 1e-15)
    assert np.unique(r.order).size == 60
    np.testing.assert_array_equal(r.idx, np.sort(r.order))


def test_permutation_equivariance():
    p, V = _data(6, 80, 32)
    perm = np.random.default_rng(0).permutation(80)
    a = greedy_select(p, V, K=30, K0=10)
    b = greedy_select(p[perm], V[perm], K=30, K0=10)
    np.testing.assert_array_equal(perm[b.order], a.order)


def test_scale_folding():
    """select(p, diag(a) V) == select(p * a, V): the raw norm belongs in the
    score.  A cosine-only residual would break this."""
    p, V = _data(7, 60, 40)
    a = np.random.default_rng(1).random(60) + 0.5
    r1 = greedy_select(p, V * a[:, None], K=25, K0=0)
    r2 = greedy_select(p * a, V, K=25, K0=0)
    np.testing.assert_array_equal(r1.order, r2.order)
    r3 = greedy_select(3.0 * p, 0.25 * V, K=25, K0=8)
    r4 = greedy_select(p, V, K=25, K0=8)
    np.testing.assert_array_equal(r3.order, r4.order)


def test_initial_basis_order_does_not_matter():
    """The span of B0 (hence every Eq. (4) residual) does not depend on the
    order R0 is orthonormalised in."""
    from oracle.select import _Basis
    p, V = _data(8, 40, 30)
    R0 = top_k0(p, 10)
    res = []
    for order in [R0, R0[::-1], np.random.default_rng(2).permutation(R0)]:
        b = _Basis(30)
        for i in order:
            b.try_append(V[i], 1e-2)
        res.append(np.linalg.norm(b.project_out(V), axis=1))
    np.testing.assert_allclose(res[1], res[0], atol=1e-12)
    np.testing.assert_allclose(res[2], res[0], atol=1e-12)


def test_rank_deficiency_falls_back_to_p_order():
    """D = 3 < K: after three independent picks every residual is zero, so the
    remaining picks follow p_hat (our total order for zero scores)."""
    rng = np.random.default_rng(9)
    V = rng.standard_normal((12, 3))
    p = rng.random(12); p /= p.sum()
    r = greedy_select(p, V, K=7, K0=1)
    assert r.appended.sum() == 3
    tail = r.order[4:]
    rest = np.setdiff1d(np.arange(12), r.order[:4])
    np.testing.assert_array_equal(tail, rest[np.argsort(-p[rest], kind="stable")[:3]])
    np.testing.assert_array_equal(r.gain[4:], 0.0)


def test_exact_duplicates_and_zero_rows():
    rng = np.random.default_rng(10)
    V = rng.standard_normal((20, 16))
    V[5] = V[2]                   # exact duplicate
    V[7] = 0.0                    # zero row
    p = np.full(20, 1.0 / 20); p[5] = p[7] = 0.2; p /= p.sum()
    r = greedy_select(p, V, K=12, K0=1)       # R0 = {5} (largest p, lower index than 7)
    assert r.order[0] == 5
    later = list(r.order[1:])
    assert 2 not in later        # V[2] == V[5] has zero residual: never beats a positive score
    assert 7 not in later        # zero row scores 0
    assert r.appended[0]


def test_restore_order():
    np.testing.assert_array_equal(restore_order([9, 2, 5]), [2, 5, 9])


def test_replay_accepts_own_order_and_rejects_planted_mistake():
    p, V = _data(11, 120, 40)
    r = greedy_select(p, V, K=40, K0=15)
    rep = replay_check(p, V, 40, 15, 1e-2, r.order, r.gain)
    assert rep.ok and rep.exact == 40 and rep.max_gain_rel_err < 1e-12
    bad = r.order.copy()
    worst = np.setdiff1d(np.arange(120), r.order)[0]
    bad[30] = worst
    rep = replay_check(p, V, 40, 15, 1e-2, bad)
    assert not rep.ok and "step 30" in rep.failure
    dup = r.order.copy(); dup[39] = dup[0]
    assert not replay_check(p, V, 40, 15, 1e-2, dup).ok


def test_replay_accepts_a_near_tie():
    """Two candidates whose scores differ by far less than the tolerance may
    come in either order."""
    rng = np.random.default_rng(12)
    Q, _ = np.linalg.qr(rng.standard_normal((16, 16)))
    V = Q[:10] * 2.0
    p = np.linspace(1.0, 0.5, 10)
    p[4] = p[3] * (1 - 1e-7)
    p /= p.sum()
    r = greedy_select(p, V, K=6, K0=0)
    assert list(r.order[3:5]) == [3, 4]
    swapped = r.order.copy(); swapped[3], swapped[4] = 4, 3
    rep = replay_check(p, V, 6, 0, 1e-2, swapped)
    assert rep.ok and rep.near_ties == 1
    assert not replay_check(p, V, 6, 0, 1e-2, swapped, tol=1e-9).ok


def test_invalid_arguments():
    p, V = _data(0, 10, 4)
    with pytest.raises(ValueError):
        greedy_select(p, V, K=11, K0=0)
    with pytest.raises(ValueError):
        greedy_select(p, V, K=3, K0=4)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_subset_selection_is_exact_when_certified(seed):
    """A greedy pick's score p n r never exceeds its bound p n.  So the
    selection run on a subset J (R0 plus the largest bounds) makes the full
    selection's picks whenever each greedy gain on J exceeds every bound
    left out -- the certificate map_prune's candidate subset relies on.
    Brute force: the full and the subset selection of small images, for
    subsets from barely past K to all tokens."""
    rng = np.random.default_rng(100 + seed)
    N, D, K, K0, tau = 160, 24, 20, 6, 1e-2
    V = rng.normal(size=(N, D)) * rng.uniform(0.5, 2.0, size=(N, 1))
    p = rng.dirichlet(np.full(N, 2.0))
    full = greedy_select(p, V, K, K0, tau)
    bound = p * np.linalg.norm(V, axis=1)
    r0 = set(top_k0(p, K0).tolist())
    by_bound = [i for i in np.lexsort((np.arange(N), -bound)) if i not in r0]
    certified = rejected = 0
    for t in range(K - K0, N - K0 + 1, 7):
        J = np.sort(np.array(sorted(r0) + by_bound[:t]))
        sub = greedy_select(p[J], V[J], K, K0, tau)
        left_out = np.setdiff1d(np.arange(N), J)
        hout = bound[left_out].max() if left_out.size else -np.inf
        if np.all(sub.gain[K0:] > hout):
            certified += 1
            np.testing.assert_array_equal(J[sub.order], full.order)
        else:
            rejected += 1
    assert certified >= 2 and rejected >= 1
