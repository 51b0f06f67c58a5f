"""Teacher selection for predictor training (section "Question Contrastive
Teacher Selection", Eq. (1)-(2); QCTS-n from the teacher-selection ablation,
Table 5).

Test infrastructure: a plain float64 statement of what the GPU path computes,
used only by the tests, the smoke check and the bench's CPU baseline.

* Eq. (1): per layer l, the text-to-vision attention A[l][h][m][n] averaged
  over the H heads and the M question tokens, then l1-normalised over the N
  visual tokens -> p^l.  The same for the reference question -> p^l_ref.
* Eq. (2): l* = argmax over layers of the Jensen-Shannon divergence
  D_JS(p^l, p^l_ref) (natural logarithm; 0 log 0 = 0).
* QCTS-n: the teacher is the mean of p^l over the n layers with the largest
  divergence (n = 1 is p^{l*}).

Readings: ties in the divergence go to the lower layer index; a layer whose
averaged attention is all zero has the uniform distribution 1/N.
"""
from dataclasses import dataclass

import numpy as np


def layer_distributions(A: np.ndarray) -> np.ndarray:
    """Eq. (1) and its l1 normalisation: A [L][H][M][N] -> p [L][N]."""
    A = np.asarray(A, dtype=np.float64)
    L, H, M, N = A.shape
    a = A.sum(axis=(1, 2)) / (H * M)                       # a_n^l, Eq. (1)
    total = a.sum(axis=1, keepdims=True)
    p = np.full((L, N), 1.0 / N)
    nz = total[:, 0] > 0
    p[nz] = a[nz] / total[nz]
    return p


def js_divergence(p: np.ndarray, q: np.ndarray) -> float:
    """Jensen-Shannon divergence of two distributions, natural logarithm."""
    p = np.asarray(p, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    m = 0.5 * (p + q)

    def kl_to_m(x):
        nz = x > 0
        return float(np.sum(x[nz] * np.log(x[nz] / m[nz])))

    return 0.5 * kl_to_m(p) + 0.5 * kl_to_m(q)


@dataclass
class TeacherResult:
    p: np.ndarray        # [L][N] question distributions p^l
    p_ref: np.ndarray    # [L][N] reference distributions p^l_ref
    js: np.ndarray       # [L] D_JS(p^l, p^l_ref)
    layers: np.ndarray   # the layers ranked by divergence, largest first (first n_top)
    teacher: np.ndarray  # [N] mean of p^l over the ranked layers


def teacher_selection(A: np.ndarray, A_ref: np.ndarray, n_top: int = 1) -> TeacherResult:
    """QCTS for one sample: A [L][H][M][N], A_ref [L][H][M_ref][N]."""
    p = layer_distributions(A)
    p_ref = layer_distributions(A_ref)
    L = p.shape[0]
    js = np.array([js_divergence(p[l], p_ref[l]) for l in range(L)])
    order = sorted(range(L), key=lambda l: (-js[l], l))   # Eq. (2); ties to the lower layer
    layers = np.array(order[:n_top], dtype=np.int32)
    teacher = p[layers].mean(axis=0)
    return TeacherResult(p, p_ref, js, layers, teacher)
