"""Pins of the PowerSGD oracle (the data-parallel compressor the paper pairs
with its method: Sec. 3.3, Sec. 5 setup, App. J family F3; Vogels et al.
2019).

Checked against what fixes the result independently of the oracle's own
code: numpy's Householder QR (positive diagonal) for the Gram-Schmidt step,
least squares for the decompressed output (the best approximation of M in
col(P_hat)), exact reconstruction of matrices of rank <= r, the rank-1
closed form, the SVD's best rank-r error (Eckart-Young) reached by the warm-
started iteration, the telescoping sum of error feedback, and brute force
for the rank of a compression ratio.  The last test plants plausible
mistakes into copies of the step and checks that these pins catch each one.
"""
import numpy as np
import pytest

from oracle import powersgd as ops
from oracle import spectral as osp


def _rng(seed):
    return np.random.default_rng(seed)


def _low_rank(m, n, k, seed, spread=(1.0, 100.0)):
    g = _rng(seed)
    U, _ = np.linalg.qr(g.standard_normal((m, k)))
    V, _ = np.linalg.qr(g.standard_normal((n, k)))
    s = np.logspace(np.log10(spread[1]), np.log10(spread[0]), k)
    return (U * s) @ V.T


def test_gram_schmidt_matches_householder_qr_with_positive_diagonal():
    P = _rng(1).standard_normal((40, 7)) @ np.diag([1, 1e-2, 3, 1e3, 1, 1e-4, 2])
    Ph = ops.gram_schmidt(P)
    Qh, R = np.linalg.qr(P)
    Qh = Qh * np.sign(np.diag(R))
    assert np.allclose(Ph, Qh, atol=1e-10)
    # P = P_hat R with R upper triangular, positive diagonal
    R2 = Ph.T @ P
    assert np.allclose(np.tril(R2, -1), 0, atol=1e-9) and np.all(np.diag(R2) > 0)
    assert np.allclose(Ph @ R2, P, atol=1e-9)


def test_gram_schmidt_drops_dependent_columns():
    a = np.array([1.0, 0.0, 0.0, 0.0])
    b = np.array([1.0, 1.0, 0.0, 0.0])
    c = np.array([0.0, 2.0, 0.0, 3.0])
    P = np.stack([a, 2 * a, b, a - b, c], axis=1)
    Ph = ops.gram_schmidt(P)
    expect = np.zeros((4, 5))
    expect[:, 0] = [1, 0, 0, 0]
    expect[:, 2] = [0, 1, 0, 0]
    expect[:, 4] = [0, 0, 0, 1]
    assert np.allclose(Ph, expect, atol=1e-12)
    assert np.array_equal(ops.gram_schmidt(np.zeros((5, 3))), np.zeros((5, 3)))


@pytest.mark.parametrize("k,r", [(1, 1), (3, 5), (8, 8)])
def test_matrices_of_rank_at_most_r_are_reconstructed_exactly(k, r):
    G = _low_rank(60, 45, k, 2 + k)
    Q = _rng(3).standard_normal((45, r))
    out = ops.step(G, np.zeros_like(G), Q)
    assert osp.rel_fro(out["out"], G) < 1e-10
    assert np.linalg.norm(out["E"]) < 1e-10 * np.linalg.norm(G)


def test_output_is_the_least_squares_fit_in_the_span_of_p_hat():
    G = _rng(4).standard_normal((50, 30))
    E = 0.1 * _rng(5).standard_normal((50, 30))
    Q = _rng(6).standard_normal((30, 4))
    o = ops.step(G, E, Q)
    X, *_ = np.linalg.lstsq(o["P_hat"], G + E, rcond=None)
    assert np.allclose(o["out"], o["P_hat"] @ X, atol=1e-10)
    # the new memory is orthogonal to the span, and energy splits (Pythagoras)
    assert np.allclose(o["P_hat"].T @ o["E"], 0, atol=1e-10)
    M = G + E
    assert abs(np.sum(M * M) - np.sum(o["out"] ** 2) - np.sum(o["E"] ** 2)) < 1e-9 * np.sum(M * M)
    assert np.linalg.matrix_rank(o["out"], tol=1e-9 * np.linalg.norm(M)) == 4


def test_rank_one_closed_form():
    G = _rng(7).standard_normal((9, 6))
    q = _rng(8).standard_normal((6, 1))
    o = ops.step(G, np.zeros_like(G), q)
    p = G @ q[:, 0]
    p = p / np.sqrt(np.sum(p * p))
    assert np.allclose(o["P_hat"][:, 0], p, atol=1e-13)
    assert np.allclose(o["Q"][:, 0], G.T @ p, atol=1e-12)
    assert np.allclose(o["out"], np.outer(p, G.T @ p), atol=1e-12)


@pytest.mark.parametrize("out_dtype", ["f64", "f32", "bf16"])
def test_error_feedback_telescopes(out_dtype):
    """E_t = E_{t-1} + G_t - out_t, so sum_t out_t + E_T = sum_t G_t + E_0:
    nothing is lost over the steps, rounding of the output included."""
    m, n, r, T = 48, 40, 3, 6
    E0 = 0.01 * _rng(9).standard_normal((m, n))
    E, Q = E0.copy(), _rng(10).standard_normal((n, r))
    sum_out, sum_g = np.zeros((m, n)), np.zeros((m, n))
    for t in range(T):
        G = _low_rank(m, n, 10, 20 + t) + 0.1 * _rng(30 + t).standard_normal((m, n))
        o = ops.step(G, E, Q, out_dtype)
        E, Q = o["E"], o["Q"]
        sum_out += o["out"]
        sum_g += G
    assert np.allclose(sum_out + E, sum_g + E0, atol=1e-11)


def test_warm_start_reaches_the_best_rank_r_error():
    """Without error feedback and with the same M every step, the warm-started
    Q makes this subspace iteration: the output tends to the best rank-r
    approximation, whose error the SVD fixes (Eckart-Young)."""
    m, n, r = 70, 50, 5
    G = _low_rank(m, n, 12, 11, spread=(1.0, 50.0))
    Q = _rng(12).standard_normal((n, r))
    for _ in range(200):
        o = ops.step(G, np.zeros_like(G), Q)
        Q = o["Q"]
    s = np.linalg.svd(G, compute_uv=False)
    best = np.sqrt(np.sum(s[r:] ** 2))
    assert abs(np.linalg.norm(G - o["out"]) - best) < 1e-8 * best
    U = np.linalg.svd(G)[0][:, :r]
    assert osp.projector_distance(o["P_hat"], U) < 1e-6


def test_rank_for_compression_ratio():
    assert ops.rank_for_ratio(8192, 8192) == 64
    assert ops.rank_for_ratio(8192, 28672) == ops.rank_for_ratio(28672, 8192) == 99
    for m, n in [(256, 256), (2048, 8192), (4096, 1024), (7, 3), (100, 100000)]:
        r = ops.rank_for_ratio(m, n)
        ok = lambda k: m * n >= 64 * k * (m + n)
        assert (ok(r) or r == 1) and not ok(r + 1)
    # a 70B-class layer compresses by at least x64 overall
    shapes = [(8192, 8192), (8192, 28672), (28672, 8192)]
    full = sum(m * n for m, n in shapes)
    sent = sum(ops.rank_for_ratio(m, n) * (m + n) for m, n in shapes)
    assert full / sent >= 64


# ----------------------------------------------------------------------------
# planted mistakes: each plausible slip in a step must fail one pin above


def _pins_hold(step):
    """The pins above, run against `step(G, E, Q) -> dict`; False at the first failure."""
    # exact reconstruction of a rank-3 matrix at r = 5
    G = _low_rank(30, 30, 3, 40)
    o = step(G, np.zeros_like(G), _rng(41).standard_normal((30, 5)))
    if osp.rel_fro(o["out"], G) > 1e-8:
        return False
    # least squares, orthonormal P_hat
    G = _rng(42).standard_normal((30, 30))
    E = 0.3 * _rng(43).standard_normal((30, 30))
    o = step(G, E, _rng(44).standard_normal((30, 4)))
    X, *_ = np.linalg.lstsq(o["P_hat"], G + E, rcond=None)
    if not np.allclose(o["out"], o["P_hat"] @ X, atol=1e-8):
        return False
    if not np.allclose(o["P_hat"].T @ o["P_hat"], np.eye(4), atol=1e-8):
        return False
    # telescoping
    E0 = 0.1 * _rng(45).standard_normal((30, 30))
    E, Q, so, sg = E0, _rng(46).standard_normal((30, 2)), 0, 0
    for t in range(3):
        G = _rng(47 + t).standard_normal((30, 30))
        o = step(G, E, Q)
        E, Q, so, sg = o["E"], o["Q"], so + o["out"], sg + G
    return bool(np.allclose(so + E, sg + E0, atol=1e-9))


def _mk(err):
    def step(G, E, Q):
        M = G + E if err != "no_feedback" else G.copy()
        P = M @ Q
        Ph = ops.gram_schmidt(P)
        if err == "no_normalise":
            Ph = Ph * np.linalg.norm(P, axis=0)
        Qn = (M @ Ph) if err == "transposed" else (M.T @ Ph)
        out = Ph @ (Q.T if err == "old_q" else Qn.T)
        Ep = (out - M) if err == "sign" else (M - out)
        if err == "memory_before_feedback":
            Ep = G - out
        return dict(P_hat=Ph, Q=Qn, out=out, E=Ep)
    return step


def test_oracle_step_passes_the_pin_harness():
    assert _pins_hold(lambda G, E, Q: ops.step(G, E, Q))
    assert _pins_hold(_mk(None))


@pytest.mark.parametrize("err", ["no_feedback", "no_normalise", "transposed", "old_q", "sign",
                                 "memory_before_feedback"])
def test_planted_mistakes_are_caught(err):
    assert not _pins_hold(_mk(err))
