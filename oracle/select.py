"""Oracle for the diversity-aware selection -- test infrastructure.

Paper, section "Inference-Time Token Pruning", Eq. (4):

1. The K0 tokens with the highest predicted attention p_hat form the initial
   retained set R0; the others are the candidates C0.
2. The embeddings of R0 are orthonormalised into an initial basis B0.
3. Until K tokens are retained, iteration t picks
       i_t = argmax_{i in C_{t-1}} p_hat_i * || v_i - B_{t-1} B_{t-1}^T v_i ||_2 ,
   moves i_t to the retained set, orthogonalises v_{i_t} against B_{t-1},
   normalises the residual and appends it, giving B_t.
4. The kept tokens are restored to their original order (their positional
   indices are kept).

Readings of what the paper leaves open (each also listed in the design notes):
* Ties: higher p_hat first in step 1; in step 3 the lower original index wins.
* R0 is orthonormalised in descending p_hat order (the span does not depend on
  the order).
* Rank deficiency: a residual with ||r|| <= tau * ||v_i|| (or v_i = 0) counts
  as zero.  Such a token adds no basis vector (it is still retained) and its
  Eq. (4) score is 0.  When every remaining candidate scores 0, the candidate
  with the highest p_hat is taken (then the lower index), so the order is total.
* The recorded gain of an R0 token is its p_hat; that of a greedy pick is its
  Eq. (4) score at the step it was taken.

Everything is float64: the residual is formed literally as v - B (B^T v) from
the current basis matrix, and a new basis vector is orthogonalised twice
(classical Gram-Schmidt with one re-orthogonalisation) before normalising.
"""
from dataclasses import dataclass, field

import numpy as np


@dataclass
class SelectResult:
    order: np.ndarray          # [K] retained tokens in selection order (R0 first)
    gain: np.ndarray           # [K] p_hat for R0 picks, Eq. (4) score for greedy picks
    idx: np.ndarray            # [K] retained tokens in ascending original order
    gaps: np.ndarray           # [K - K0] relative decisive gap of each greedy step
    appended: np.ndarray       # [K] whether the pick added a basis vector


class _Basis:
    """Orthonormal columns B [D, k] spanning the retained embeddings."""

    def __init__(self, D: int):
        self.D = D
        self.cols = []
        self._B = np.zeros((D, 0))

    def project_out(self, X: np.ndarray) -> np.ndarray:
        """X - (X B) B^T for rows X [n, D]."""
        if not self.cols:
            return X.copy()
        return X - (X @ self._B) @ self._B.T

    def try_append(self, v: np.ndarray, tau: float) -> bool:
        nv = np.linalg.norm(v)
        r = self.project_out(v[None, :])
        r = self.project_out(r)[0]                 # second orthogonalisation pass
        nr = np.linalg.norm(r)
        if nv == 0.0 or nr <= tau * nv:
            return False
        self.cols.append(r / nr)
        self._B = np.stack(self.cols, axis=1)
        return True


def _scores(p, V, basis: _Basis, tau: float, vnorm: np.ndarray) -> np.ndarray:
    """Eq. (4) score p_hat_i * ||v_i - B B^T v_i|| of every token (0 below tau)."""
    rn = np.linalg.norm(basis.project_out(V), axis=1)
    alive = (vnorm > 0) & (rn > tau * vnorm)
    return np.where(alive, p * rn, 0.0)


def _best(cands: np.ndarray, s: np.ndarray, p: np.ndarray) -> int:
    """Candidate with the largest key (s > 0, s or p_hat, lower index)."""
    cs = s[cands]
    if np.any(cs > 0):
        return int(cands[np.argmax(cs)])          # argmax takes the first, i.e. lowest, index
    return int(cands[np.argmax(p[cands])])


def _rel_gap(cands: np.ndarray, s: np.ndarray, p: np.ndarray, best: int) -> float:
    """Relative gap between the best and the runner-up key at one decision."""
    rest = cands[cands != best]
    if rest.size == 0:
        return np.inf
    if s[best] > 0:
        return float((s[best] - s[rest].max()) / s[best])
    pb = p[best]
    return float((pb - p[rest].max()) / pb) if pb > 0 else 0.0


def top_k0(p, K0: int) -> np.ndarray:
    """R0: the K0 tokens with the largest p_hat, in descending p_hat order
    (ties: lower index first)."""
    p = np.asarray(p, np.float64)
    order = np.lexsort((np.arange(p.size), -p))
    return order[:K0].astype(np.int64)


def restore_order(order) -> np.ndarray:
    """Kept tokens back in their original (ascending) order."""
    return np.sort(np.asarray(order, np.int64))


def greedy_select(p, V, K: int, K0: int, tau: float = 1e-2) -> SelectResult:
    """Selection of one image: p [N] importance, V [N, D] raw embeddings."""
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    N, D = V.shape
    if not (0 <= K0 <= K <= N):
        raise ValueError("need 0 <= K0 <= K <= N")
    vnorm = np.linalg.norm(V, axis=1)
    basis = _Basis(D)
    selected = np.zeros(N, bool)
    order, gain, appended, gaps = [], [], [], []
    for i in top_k0(p, K0):
        selected[i] = True
        order.append(int(i))
        gain.append(p[i])
        appended.append(basis.try_append(V[i], tau))
    for _ in range(K0, K):
        s = _scores(p, V, basis, tau, vnorm)
        cands = np.flatnonzero(~selected)
        i = _best(cands, s, p)
        gaps.append(_rel_gap(cands, s, p, i))
        selected[i] = True
        order.append(i)
        gain.append(s[i])
        appended.append(basis.try_append(V[i], tau))
    order = np.asarray(order, np.int64)
    return SelectResult(order=order, gain=np.asarray(gain), idx=restore_order(order),
                        gaps=np.asarray(gaps), appended=np.asarray(appended, bool))


@dataclass
class ReplayReport:
    ok: bool
    steps: int = 0
    exact: int = 0                 # picks equal to the oracle's own argmax
    near_ties: int = 0             # accepted picks within the tolerance of the argmax
    max_gain_rel_err: float = 0.0  # |gain - oracle score| / oracle score over greedy picks
    min_gap: float = np.inf        # smallest decisive gap met along the replay
    failure: str = ""
    details: list = field(default_factory=list)


def replay_check(p, V, K: int, K0: int, tau: float, order, gain=None,
                 tol: float = 1e-4) -> ReplayReport:
    """Check another implementation's selection order against the oracle.

    Each decision is replayed on the other side's own prefix: a pick is
    accepted when it is the oracle's choice at that point, or when its key
    lies within a relative ``tol`` of the oracle's best key (the decisive gap
    there is below ``tol``, so either choice is correct to that precision).
    ``gain`` (optional) is compared with the oracle's score of each greedy pick.
    """
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    order = np.asarray(order, np.int64)
    N, D = V.shape
    rep = ReplayReport(ok=False)
    if order.shape != (K,):
        rep.failure = f"order has shape {order.shape}, expected ({K},)"
        return rep
    if np.any(order < 0) or np.any(order >= N) or np.unique(order).size != K:
        rep.failure = "order holds out-of-range or repeated indices"
        return rep
    vnorm = np.linalg.norm(V, axis=1)
    selected = np.zeros(N, bool)
    basis = _Basis(D)
    for t in range(K):
        got = int(order[t])
        cands = np.flatnonzero(~selected)
        if t < K0:
            exp = int(cands[np.argmax(p[cands])])
            ok = got == exp or p[got] >= (1.0 - tol) * p[exp]
            key_got, key_exp = p[got], p[exp]
        else:
            s = _scores(p, V, basis, tau, vnorm)
            exp = _best(cands, s, p)
            gap = _rel_gap(cands, s, p, exp)
            rep.min_gap = min(rep.min_gap, gap)
            if s[exp] > 0:
                ok = got == exp or s[got] >= (1.0 - tol) * s[exp]
                key_got, key_exp = s[got], s[exp]
            else:
                ok = got == exp or (s[got] == 0 and p[got] >= (1.0 - tol) * p[exp])
                key_got, key_exp = p[got], p[exp]
            if gain is not None and s[got] > 0:
                rel = abs(float(gain[t]) - s[got]) / s[got]
                rep.max_gain_rel_err = max(rep.max_gain_rel_err, rel)
        rep.steps += 1
        if got == exp:
            rep.exact += 1
        elif ok:
            rep.near_ties += 1
            rep.details.append((t, got, exp, float(key_got), float(key_exp)))
        else:
            rep.failure = (f"step {t}: picked {got} (key {key_got:.9g}) but the oracle's "
                           f"best is {exp} (key {key_exp:.9g})")
            return rep
        selected[got] = True
        basis.try_append(V[got], tau)
    rep.ok = True
    return rep
