"""PowerSGD compressor with error feedback, one worker's share, float64 numpy.

TEST INFRASTRUCTURE ONLY.  The paper pairs its pipeline-side method with
PowerSGD (Vogels, Karimireddy & Jaggi 2019) at x64 compression on the
data-parallel side (Sec. 2 related work, Sec. 3.3, Sec. 5 setup; App. J,
family F3: a low-rank sketch by subspace iteration, linear so that it
commutes with the all-reduce, with error feedback).  This module is that
compressor's definition, one step per function, written from the published
algorithm:

  error feedback      M = G + E                          (E: the worker's memory)
  project             P = M Q                            (Q: previous step's Q)
  orthogonalise       P_hat = Gram-Schmidt(P)            (columns in order)
  project back        Q' = M^T P_hat
  decompress          out = P_hat Q'^T                   (rank <= r)
  memory              E' = M - out                       (what the output lost)

The two all-reduces of the algorithm (of P before the Gram-Schmidt, of Q'
after the second projection) are means over the data-parallel workers; on one
worker they are the identity, so they do not appear here.  Q' is the next
step's Q (warm start).

Readings (the cited algorithm leaves them open): Gram-Schmidt drops a column
whose residual is numerically zero (squared norm at or below
1e-15 * r * max_i ||P_i||^2), leaving a zero column, so that P_hat's nonzero
columns are an orthonormal basis of col(P); the output is rounded to its
storage type (bf16 or fp32) and the memory is taken against the rounded
output, so that what the output loses to rounding is fed back too; the rank
of a matrix for a compression ratio rho is the largest r with
m n / (r (m + n)) >= rho (factors P and Q carried in the gradient's type),
at least 1.
"""
from __future__ import annotations

import math

import numpy as np
import torch

DROP = 1e-15


def rank_for_ratio(m: int, n: int, ratio: float = 64.0) -> int:
    """Largest r with m n / (r (m + n)) >= ratio, at least 1."""
    return max(1, int(math.floor(m * n / (ratio * (m + n)))))


def gram_schmidt(P: np.ndarray) -> np.ndarray:
    """P_hat: columns of P orthonormalised in order (each column made
    orthogonal to the kept earlier ones, twice, then normalised); a column
    with a numerically zero residual becomes a zero column."""
    P = np.asarray(P, dtype=np.float64)
    m, r = P.shape
    out = np.zeros((m, r))
    scale = max(float(np.max(np.sum(P * P, axis=0))) if r else 0.0, 0.0)
    thresh = DROP * r * scale
    for j in range(r):
        v = P[:, j].copy()
        for _ in range(2):                      # re-orthogonalise ("twice is enough")
            for i in range(j):
                v -= (out[:, i] @ v) * out[:, i]
        nn = float(v @ v)
        if nn > thresh and nn > 0.0:
            out[:, j] = v / math.sqrt(nn)
    return out


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """x rounded to the output's storage type (via fp32, nearest even), as float64."""
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    t = torch.from_numpy(np.asarray(x, dtype=np.float64)).float()
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    elif dtype != "f32":
        raise ValueError(dtype)
    return t.double().numpy()


def project(G: np.ndarray, E: np.ndarray, Q: np.ndarray):
    """First half: M = G + E and P = M Q."""
    M = np.asarray(G, dtype=np.float64) + np.asarray(E, dtype=np.float64)
    return M, M @ np.asarray(Q, dtype=np.float64)


def step(G, E, Q, out_dtype: str = "f64"):
    """One PowerSGD step with error feedback on one worker.

    G [m, n], E [m, n] (memory), Q [n, r] (previous Q).  Returns a dict with
    M, P (before orthogonalisation), P_hat, Q (the new Q'), out and E (the
    new memory E' = M - out).
    """
    M, P = project(G, E, Q)
    P_hat = gram_schmidt(P)
    Qn = M.T @ P_hat
    out = round_to(P_hat @ Qn.T, out_dtype)
    return dict(M=M, P=P, P_hat=P_hat, Q=Qn, out=out, E=M - out)

