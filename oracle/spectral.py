"""Spectral-correction oracle (paper Sec. 3.2; Alg. 1; App. E), float64 numpy.

TEST INFRASTRUCTURE ONLY.  Plain definitions, one step per function, in the
order and notation of the paper:

  anchor EMA          M <- beta * M + (1 - beta) * G_anc          (Sec. 3.2 eq.)
  SVD of the EMA      M = U S V^T, truncated to the top r triplets  (Sec. 3.2; App. E)
  soft filter         d_i = s_i / (s_i + tau)                      (Sec. 3.2 eq.)
  two-sided filter    X = U^T G V;  X_f = diag(d) X diag(d);
                      G_filt = U X_f V^T                           (Sec. 3.2)
  blend               G_proj = alpha * G + (1 - alpha) * G_filt    (Sec. 3.2 eq.)

Readings of the paper taken here (the paper does not fix them):
  * the top-r truncation of App. E, applied before the soft filter;
  * tau acts on the raw singular values of the EMA;
  * 0 / 0 in the filter (s_i = 0 with tau = 0) is taken as d_i = 0, so an
    empty prior (M = 0) gives G_proj = alpha * G.
The SVD is LAPACK's (numpy.linalg.svd), a library primitive.  For matrices
whose full SVD would take minutes on the host, ``top_r_svd_gram`` reaches the
same top-r triplets through the symmetric eigendecomposition of the smaller
Gram matrix (LAPACK's dsyevr, also a library primitive).
"""
from __future__ import annotations

import numpy as np
import scipy.linalg


def ema(M_prev: np.ndarray, G_anc: np.ndarray, beta: float) -> np.ndarray:
    """Anchor-momentum EMA, one arrival (Sec. 3.2 eq.; Alg. 1)."""
    return beta * np.asarray(M_prev, dtype=np.float64) + (1.0 - beta) * np.asarray(G_anc, dtype=np.float64)


def top_r_svd(M: np.ndarray, r: int):
    """Top-r singular triplets of M (Sec. 3.2; App. E truncation).

    Returns U [m, r], s [r] (descending), V [n, r]."""
    M = np.asarray(M, dtype=np.float64)
    U, s, Vt = np.linalg.svd(M, full_matrices=False)
    return U[:, :r].copy(), s[:r].copy(), Vt[:r, :].T.copy()


def top_r_svd_gram(M: np.ndarray, r: int):
    """Top-r singular triplets of M (Sec. 3.2; App. E truncation) from the
    Gram matrix of its shorter side.

    For m <= n, M M^T = U S^2 U^T: the r largest eigenpairs give U and s, and
    V = M^T U S^-1 (column i is M^T u_i / s_i).  For m > n the roles swap
    through M^T M = V S^2 V^T.  A zero singular value leaves a zero column on
    the derived side.  Returns U [m, r], s [r] (descending), V [n, r]."""
    M = np.asarray(M, dtype=np.float64)
    m, n = M.shape
    wide = m <= n
    A = M @ M.T if wide else M.T @ M
    k = A.shape[0]
    w, X = scipy.linalg.eigh(A, subset_by_index=[k - r, k - 1], driver="evr")
    order = np.argsort(w)[::-1]
    w, X = np.maximum(w[order], 0.0), X[:, order]
    s = np.sqrt(w)
    Y = M.T @ X if wide else M @ X
    inv = np.zeros_like(s)
    inv[s > 0] = 1.0 / s[s > 0]
    Y = Y * inv
    return (X, s, Y) if wide else (Y, s, X)


def filter_weights(s: np.ndarray, tau: float) -> np.ndarray:
    """d_i = s_i / (s_i + tau) (Sec. 3.2 eq.), with 0/0 read as 0."""
    s = np.asarray(s, dtype=np.float64)
    den = s + tau
    d = np.zeros_like(s)
    nz = den != 0
    d[nz] = s[nz] / den[nz]
    return d


def two_sided_filter(G: np.ndarray, U: np.ndarray, d: np.ndarray, V: np.ndarray) -> np.ndarray:
    """G_filt = U diag(d) (U^T G V) diag(d) V^T (Sec. 3.2; App. E P_t)."""
    G = np.asarray(G, dtype=np.float64)
    X = U.T @ G @ V
    Xf = d[:, None] * X * d[None, :]
    return U @ Xf @ V.T


def correct(G: np.ndarray, U: np.ndarray, d: np.ndarray, V: np.ndarray, alpha: float) -> np.ndarray:
    """G_proj = alpha * G + (1 - alpha) * G_filt (Sec. 3.2 eq.; Alg. 1)."""
    G = np.asarray(G, dtype=np.float64)
    return alpha * G + (1.0 - alpha) * two_sided_filter(G, U, d, V)


def correct_rows(G, U: np.ndarray, d: np.ndarray, V: np.ndarray, alpha: float, rows) -> np.ndarray:
    """Rows `rows` of G_proj = alpha G + (1 - alpha) U diag(d) (U^T G V) diag(d)
    V^T (Sec. 3.2 eq.; Alg. 1), for matrices too large to form G_proj whole.

    X = U^T (G V) needs all of G; it is accumulated in float64 over blocks of
    rows of G (an array or a callable giving rows [a, b) as an array)."""
    m = U.shape[0]
    get = G if callable(G) else (lambda a, b: np.asarray(G[a:b], dtype=np.float64))
    X = np.zeros((U.shape[1], V.shape[1]))
    for a in range(0, m, 1024):
        b = min(m, a + 1024)
        X += U[a:b].T @ (get(a, b) @ V)
    Xf = d[:, None] * X * d[None, :]
    rows = np.asarray(rows)
    Gr = np.concatenate([get(int(i), int(i) + 1) for i in rows], axis=0)
    return alpha * Gr + (1.0 - alpha) * (U[rows] @ Xf @ V.T)


def build_prior(M_prev, G_anc, beta: float, r: int, tau: float):
    """EMA (if an anchor gradient arrived), then top-r SVD and filter weights.

    Returns (M, U, s, V, d)."""
    M = ema(M_prev, G_anc, beta) if G_anc is not None else np.asarray(M_prev, dtype=np.float64)
    U, s, V = top_r_svd(M, r)
    d = filter_weights(s, tau)
    return M, U, s, V, d


def corrected_step(M_prev, G_anc, G_mask, beta: float, r: int, tau: float, alpha: float):
    """One pass of the corrector for one matrix: build the prior, then correct."""
    M, U, s, V, d = build_prior(M_prev, G_anc, beta, r, tau)
    return M, U, s, V, d, correct(G_mask, U, d, V, alpha)


def alignment(g: np.ndarray, U: np.ndarray, V: np.ndarray) -> float:
    """eta_r = ||U^T g V||_F^2 / ||g||_F^2 (App. G)."""
    g = np.asarray(g, dtype=np.float64)
    num = np.linalg.norm(U.T @ g @ V) ** 2
    den = np.linalg.norm(g) ** 2
    return float(num / den) if den > 0 else 0.0


def projector_distance(U1: np.ndarray, U2: np.ndarray, method: str = "auto") -> float:
    """||U1 U1^T - U2 U2^T||_F / sqrt(2 r): basis-free subspace distance.

    "projector" forms the two m x m projectors.  "residual" (the default past
    m = 4096, where those would take gigabytes) uses, for orthonormal bases
    of equal rank at principal angles theta_i,
    ||P1 - P2||_F^2 = 2 sum sin^2 theta_i = 2 ||U1 - U2 (U2^T U1)||_F^2."""
    r = U1.shape[1]
    if method == "auto":
        method = "projector" if U1.shape[0] <= 4096 else "residual"
    if method == "projector":
        P1 = U1 @ U1.T
        P2 = U2 @ U2.T
        return float(np.linalg.norm(P1 - P2) / np.sqrt(2.0 * r))
    return float(np.linalg.norm(U1 - U2 @ (U2.T @ U1)) / np.sqrt(r))


def rel_fro(a, b) -> float:
    """||a - b||_F / ||b||_F."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a - b))
