"""Corrected AdamW step oracle, float64 numpy (paper Alg. 1: the fast weights
are updated by AdamW on G_proj; App. I: AdamW with (beta1, beta2) =
(0.9, 0.999) and the gradient norm clipped at 0.2).

TEST INFRASTRUCTURE ONLY.  Plain definitions, one step per function:

  global norm         N = sqrt(sum over the call's matrices of ||G_proj||_F^2)
  clipping            c = min(1, max_norm / (N + 1e-6)),  g = c * G_proj
                      (global-norm clipping, Pascanu, Mikolov & Bengio 2013)
  AdamW, step t >= 1  (decoupled weight decay, Loshchilov & Hutter 2019)
                      W <- W (1 - lr * wd)
                      m <- beta1 m + (1 - beta1) g
                      v <- beta2 v + (1 - beta2) g^2
                      W <- W - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)

G_proj itself is spectral.correct (Sec. 3.2 eq.; Alg. 1).

Readings (the paper does not fix them): eps and the 1e-6 guard of the
clipping ratio are arguments, defaulting to the values of the common PyTorch
implementation (1e-8, 1e-6); the weight decay is an argument (the SFT runs
state none); max_norm <= 0 means no clipping; the norm is taken over the
matrices of one call (on one pipeline stage, the stage's targeted matrices).
"""
from __future__ import annotations

import numpy as np

from . import spectral as osp

CLIP_GUARD = 1e-6


def global_norm(grads) -> float:
    """N = sqrt(sum_i ||g_i||_F^2) over every gradient of the call."""
    return float(np.sqrt(sum(float(np.sum(np.asarray(g, dtype=np.float64) ** 2)) for g in grads)))


def clip_coefficient(norm: float, max_norm: float, guard: float = CLIP_GUARD) -> float:
    """Scale of global-norm clipping: min(1, max_norm / (N + guard)); 1 when max_norm <= 0."""
    if max_norm <= 0:
        return 1.0
    return min(1.0, max_norm / (norm + guard))


def adamw(W, m, v, g, lr: float, beta1: float, beta2: float, eps: float, weight_decay: float, t: int):
    """One AdamW step at step t >= 1 on gradient g; returns the new (W, m, v)."""
    W = np.asarray(W, dtype=np.float64)
    m = np.asarray(m, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    W = W * (1.0 - lr * weight_decay)
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    W = W - lr * m_hat / (np.sqrt(v_hat) + eps)
    return W, m, v


def corrected_adamw(mats, alpha: float, lr: float, beta1: float, beta2: float, eps: float,
                    weight_decay: float, t: int, max_norm: float):
    """Alg. 1's correction then update for every matrix of one call.

    mats: sequence of dicts with G, U, d, V (the prior) and W, m, v (the
    optimiser state).  Returns ([(W, m, v) per matrix], N) with N the global
    norm of the G_proj before clipping."""
    gp = [osp.correct(x["G"], x["U"], x["d"], x["V"], alpha) for x in mats]
    N = global_norm(gp)
    c = clip_coefficient(N, max_norm)
    out = [adamw(x["W"], x["m"], x["v"], c * g, lr, beta1, beta2, eps, weight_decay, t)
           for x, g in zip(mats, gp)]
    return out, N
