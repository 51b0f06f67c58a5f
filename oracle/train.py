"""Oracle for one predictor training step -- test infrastructure.

Paper, section "Cross-Modal Attention Distillation": offline, the predictor
is trained by minimising the Kullback-Leibler divergence from the teacher
layer's attention distribution p^{l*} (Eq. (1)-(2)) to the predicted
distribution p_hat of Eq. (3):

    loss = D_KL(p^{l*} || p_hat) = sum_n p*_n log(p*_n / p_hat_n)   (0 log 0 = 0)

The step computes this loss and its gradient with respect to every
predictor parameter: f_V = (W1_v, b1_v, W2_v, b2_v), f_T = (W1_t, b1_t,
W2_t, b2_t), W_K and W_Q.  The inputs V, T (the frozen multimodal features)
receive no gradient.

Readings of what the paper leaves open (each also listed in the design
notes):
* For a batch of images the objective is the mean of the per-image
  divergences (the batch's images weigh equally).
* The natural logarithm.  The teacher rows must be distributions over the
  N visual tokens (non-negative, summing to one).
* The predictor is the one of Eq. (3) as read in ``predictor``: two-layer
  GELU(erf) MLPs, a single head of width d, RoPE on queries and keys,
  softmax over the visual tokens, mean over the question tokens.

The gradient is the chain rule written out step by step, in the order the
forward pass runs backwards, in float64:

    dL/dp_hat_n   = -p*_n / p_hat_n / B
    dL/dP_mn      = dL/dp_hat_n / M                (p_hat = mean_m P_m)
    dL/dl_mn      = P_mn (dL/dP_mn - sum_n' P_mn' dL/dP_mn')   (softmax)
    dL/dq_m       = sum_n dL/dl_mn k_n / sqrt(d),  dL/dk_n = sum_m dL/dl_mn q_m / sqrt(d)
    RoPE is a rotation per pair: its transpose rotates by the opposite angle
    dL/dW_Q       = sum_m dq~_m u_m^T,  dL/du_m = W_Q^T dq~_m     (u = f_T(t))
    dL/dW2, db2   = sum_m du_m h_m^T, sum_m du_m;   dL/dh_m = W2^T du_m
    dL/da_m       = dL/dh_m * GELU'(a_m),  GELU'(x) = Phi(x) + x phi(x)
    dL/dW1, db1   = sum_m da_m t_m^T, sum_m da_m
and the same on the visual side with k, W_K and f_V.  Matrix products are
library primitives; nothing is fused or reassociated.
"""
from dataclasses import dataclass

import numpy as np
from scipy.special import erf

from .predictor import gelu_erf, rope

PARAMS = ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")


def gelu_erf_grad(x: np.ndarray) -> np.ndarray:
    """d/dx [x Phi(x)] = Phi(x) + x phi(x)."""
    x = np.asarray(x, np.float64)
    return 0.5 * (1.0 + erf(x / np.sqrt(2.0))) + x * np.exp(-0.5 * x * x) / np.sqrt(2.0 * np.pi)


def kl_divergence(p_star, p_hat) -> float:
    """D_KL(p* || p_hat) with the natural log and 0 log 0 = 0."""
    p_star = np.asarray(p_star, np.float64)
    p_hat = np.asarray(p_hat, np.float64)
    nz = p_star > 0
    return float(np.sum(p_star[nz] * np.log(p_star[nz] / p_hat[nz])))


def _branch_forward(X, w1, b1, w2, b2, wp, pos, theta):
    a = X @ w1.T + b1            # layer 1 pre-activation
    h = gelu_erf(a)
    u = h @ w2.T + b2            # f(X)
    z = u @ wp.T                 # projection (W_Q or W_K), before RoPE
    return a, h, u, rope(z, pos, theta)


def _branch_backward(X, a, h, u, w2, wp, dz, g, s):
    """Gradients of one branch given dL/dz (z: the projection before RoPE);
    g, s name the branch's parameters ('t', 'q') or ('v', 'k')."""
    du = dz @ wp                 # dL/du = W^T dz, row-wise
    dh = du @ w2                 # dL/dh = W2^T du
    da = dh * gelu_erf_grad(a)
    return {f"w_{s}": dz.T @ u, f"w2_{g}": du.T @ h, f"b2_{g}": du.sum(axis=0),
            f"w1_{g}": da.T @ X, f"b1_{g}": da.sum(axis=0)}


def image_loss_and_grads(V, T, pos_v, pos_t, w: dict, p_star, theta: float = 10000.0, scale: float = 1.0):
    """One image: (loss, p_hat, grads of scale * loss) for V [N, D], T [M, D]."""
    V = np.asarray(V, np.float64)
    T = np.asarray(T, np.float64)
    g = {k: np.asarray(v, np.float64) for k, v in w.items()}
    p_star = np.asarray(p_star, np.float64)
    av, hv, uv, k = _branch_forward(V, g["w1_v"], g["b1_v"], g["w2_v"], g["b2_v"], g["w_k"], pos_v, theta)
    at, ht, ut, q = _branch_forward(T, g["w1_t"], g["b1_t"], g["w2_t"], g["b2_t"], g["w_q"], pos_t, theta)
    M, d = q.shape
    logits = q @ k.T / np.sqrt(d)                                  # [M, N]
    e = np.exp(logits - logits.max(axis=1, keepdims=True))
    P = e / e.sum(axis=1, keepdims=True)                           # softmax over n
    p_hat = P.mean(axis=0)
    loss = kl_divergence(p_star, p_hat)
    # backward
    dp = np.where(p_star > 0, -p_star / p_hat, 0.0) * scale        # dL/dp_hat
    dP = np.broadcast_to(dp / M, P.shape)                          # mean over m
    dl = P * (dP - (P * dP).sum(axis=1, keepdims=True))            # softmax backward
    dq = dl @ k / np.sqrt(d)
    dk = dl.T @ q / np.sqrt(d)
    dzq = rope(dq, -np.asarray(pos_t, np.float64), theta)          # R(pos)^T = R(-pos)
    dzk = rope(dk, -np.asarray(pos_v, np.float64), theta)
    grads = _branch_backward(T, at, ht, ut, g["w2_t"], g["w_q"], dzq, "t", "q")
    grads.update(_branch_backward(V, av, hv, uv, g["w2_v"], g["w_k"], dzk, "v", "k"))
    return loss, p_hat, grads


@dataclass
class TrainStepResult:
    loss: float            # mean over the batch's images of D_KL(p* || p_hat)
    image_loss: np.ndarray  # [B] each image's D_KL
    p_hat: np.ndarray      # [B, N]
    grads: dict            # parameter name -> gradient of `loss` (float64, the parameter's shape)


def train_step(V, T, t_off, pos_v, pos_t, w: dict, p_teacher, theta: float = 10000.0) -> TrainStepResult:
    """Loss and gradients of one batch: V [B, N, D], T [sum M, D] with
    offsets t_off [B + 1], teacher distributions p_teacher [B, N]."""
    V = np.asarray(V)
    B, N, _ = V.shape
    grads = {k: np.zeros(np.shape(w[k])) for k in PARAMS}
    losses = np.empty(B)
    p_hat = np.empty((B, N))
    for b in range(B):
        lo, hi = int(t_off[b]), int(t_off[b + 1])
        losses[b], p_hat[b], gb = image_loss_and_grads(V[b], T[lo:hi], pos_v[b], pos_t[lo:hi], w, p_teacher[b],
                                                       theta, scale=1.0 / B)
        for k in PARAMS:
            grads[k] += gb[k]
    return TrainStepResult(float(losses.mean()), losses, p_hat, grads)
