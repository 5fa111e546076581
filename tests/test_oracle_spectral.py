"""Pins of the spectral-correction oracle (paper Sec. 3.2; Alg. 1; App. E).

The oracle is checked against things other than itself: closed forms for
inputs whose SVD is known by construction, the special cases the paper names
(alpha = 1; the filter never amplifies), projector identities at tau = 0,
Lemma 1 (non-expansive), Lemma 2 (expected noise contraction, by Monte
Carlo), the EMA's closed form, and a different LAPACK routine (eigh) for the
singular values.  The last test plants plausible mistakes into the oracle and
checks that these pins catch each of them.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import spectral as osp


def _basis(m, n, r, seed):
    U, s, V = workloads.random_orthonormal_basis(m, n, r, seed)
    return U.numpy(), s.numpy(), V.numpy()


def _closed_form_case(m=40, n=28, rho=6, seed=0):
    U, s, V = _basis(m, n, rho, seed)
    M = (U * s) @ V.T
    return M, U, s, V


@pytest.mark.parametrize("r", [6, 3])
def test_closed_form_when_gradient_equals_the_prior(r):
    # G = M = U S V^T  =>  G_proj = alpha G + (1-alpha) U_r diag(d_i^2 s_i) V_r^T
    M, U, s, V = _closed_form_case()
    alpha, tau = 0.3, 1.0          # tau of the order of s so that d spreads in (0, 1)
    Uo, so, Vo = osp.top_r_svd(M, r)
    do = osp.filter_weights(so, tau)
    got = osp.correct(M, Uo, do, Vo, alpha)
    d_true = s[:r] / (s[:r] + tau)
    expect = alpha * M + (1 - alpha) * (U[:, :r] * (d_true ** 2 * s[:r])) @ V[:, :r].T
    assert np.allclose(got, expect, rtol=0, atol=1e-12 * np.abs(M).max())
    if r == 6:
        # full rank of the signal: diag((alpha + (1-alpha) d^2) s)
        expect2 = (U * ((alpha + (1 - alpha) * d_true ** 2) * s)) @ V.T
        assert np.allclose(got, expect2, rtol=0, atol=1e-12 * np.abs(M).max())


def test_svd_recovers_constructed_singular_values_and_subspaces():
    M, U, s, V = _closed_form_case(60, 45, 7, 3)
    Uo, so, Vo = osp.top_r_svd(M, 7)
    assert np.allclose(so, s, rtol=1e-12)
    assert np.all(np.diff(so) <= 0) and np.all(so >= 0)
    assert np.allclose(Uo.T @ Uo, np.eye(7), atol=1e-12)
    assert np.allclose(Vo.T @ Vo, np.eye(7), atol=1e-12)
    assert osp.projector_distance(Uo, U) < 1e-10
    assert osp.projector_distance(Vo, V) < 1e-10


@pytest.mark.parametrize("m,n", [(30, 50), (50, 30), (64, 64)])
def test_singular_values_agree_with_eigh_of_the_gram_matrix(m, n):
    rng = np.random.default_rng(m * 7 + n)
    M = rng.standard_normal((m, n))
    r = 5
    Uo, so, Vo = osp.top_r_svd(M, r)
    small = M @ M.T if m <= n else M.T @ M
    ev = np.linalg.eigh(small)[0][::-1][:r]
    assert np.allclose(so ** 2, ev, rtol=1e-10)
    # singular triplets: M v = s u and M^T u = s v
    assert np.allclose(M @ Vo, Uo * so, atol=1e-10)
    assert np.allclose(M.T @ Uo, Vo * so, atol=1e-10)


def test_alpha_one_recovers_masked_only_training():
    rng = np.random.default_rng(1)
    G = rng.standard_normal((33, 21))
    U, s, V = _basis(33, 21, 4, 9)
    d = osp.filter_weights(s, 1e-3)
    assert np.array_equal(osp.correct(G, U, d, V, 1.0), G)


def test_filter_weights_lie_in_unit_interval_and_zero_prior_gives_alpha_G():
    s = np.array([0.0, 1e-6, 1e-3, 1.0, 1e6])
    d = osp.filter_weights(s, 1e-3)
    assert np.all(d >= 0) and np.all(d < 1)
    assert d[0] == 0 and abs(d[2] - 0.5) < 1e-15
    # M = 0 (no anchor arrived yet): d = 0 so G_proj = alpha * G
    G = np.random.default_rng(2).standard_normal((12, 9))
    M, U, s0, V, d0 = osp.build_prior(np.zeros((12, 9)), None, 0.9, 3, 1e-3)
    assert np.all(d0 == 0)
    assert np.allclose(osp.correct(G, U, d0, V, 0.3), 0.3 * G)
    assert np.all(osp.filter_weights(np.zeros(3), 0.0) == 0)


def test_tau_zero_filter_is_an_orthogonal_projector():
    U, s, V = _basis(26, 19, 5, 4)
    d = osp.filter_weights(s, 0.0)
    assert np.allclose(d, 1.0)
    rng = np.random.default_rng(5)
    A = rng.standard_normal((26, 19))
    B = rng.standard_normal((26, 19))
    P = lambda X: osp.correct(X, U, d, V, 0.0)
    assert np.allclose(P(P(A)), P(A), atol=1e-12)                       # idempotent
    assert abs(np.sum(P(A) * B) - np.sum(A * P(B))) < 1e-10             # self-adjoint


def test_gradient_orthogonal_to_the_left_basis_is_filtered_out():
    U, s, V = _basis(31, 17, 4, 6)
    rng = np.random.default_rng(7)
    N = rng.standard_normal((31, 17))
    G = N - U @ (U.T @ N)
    d = osp.filter_weights(s, 1e-3)
    assert np.abs(osp.two_sided_filter(G, U, d, V)).max() < 1e-12
    H = N - (N @ V) @ V.T                                                # right side too
    assert np.abs(osp.two_sided_filter(H, U, d, V)).max() < 1e-12


def test_lemma1_non_expansive():
    rng = np.random.default_rng(8)
    for t in range(20):
        m, n, r = 20 + t, 35 - t, 1 + t % 6
        U, s, V = _basis(m, n, r, 100 + t)
        d = osp.filter_weights(s, 10 ** rng.uniform(-3, 1))
        G = rng.standard_normal((m, n)) * rng.uniform(0.1, 10)
        Pg = osp.two_sided_filter(G, U, d, V)
        assert np.linalg.norm(Pg) <= np.linalg.norm(G) * (1 + 1e-12)
        # tight case: G inside span(U) x span(V) gives ||P G|| = ||d^2 * c||
        c = rng.standard_normal(r)
        Gin = (U * c) @ V.T
        Pin = osp.two_sided_filter(Gin, U, d, V)
        assert np.linalg.norm(Pin) <= np.linalg.norm(Gin) * (1 + 1e-12)
        assert abs(np.linalg.norm(Pin) - np.linalg.norm(d ** 2 * c)) < 1e-12 * np.linalg.norm(c)


def test_lemma2_noise_contraction_monte_carlo():
    # E ||P eps||_F^2 = sigma^2 (sum d_i^2)_U (sum d_i^2)_V / (m n) for iid eps
    # with E[vec vec^T] = sigma^2/(mn) I
    m, n, r, trials, sigma2 = 24, 16, 4, 4000, 3.0
    U, s, V = _basis(m, n, r, 11)
    d = osp.filter_weights(s, 1.5)
    rng = np.random.default_rng(12)
    vals = np.empty(trials)
    for t in range(trials):
        eps = rng.standard_normal((m, n)) * np.sqrt(sigma2 / (m * n))
        vals[t] = np.linalg.norm(osp.two_sided_filter(eps, U, d, V)) ** 2
    theory = sigma2 * np.sum(d ** 2) ** 2 / (m * n)
    se = vals.std() / np.sqrt(trials)
    assert abs(vals.mean() - theory) < 5 * se, (vals.mean(), theory, se)


def test_sign_flips_of_singular_pairs_leave_the_correction_unchanged():
    U, s, V = _basis(22, 30, 5, 13)
    d = osp.filter_weights(s, 0.7)
    G = np.random.default_rng(14).standard_normal((22, 30))
    flip = np.array([1, -1, 1, -1, -1.0])
    a = osp.correct(G, U, d, V, 0.3)
    b = osp.correct(G, U * flip, d, V * flip, 0.3)
    assert np.allclose(a, b, atol=1e-13)


def test_ema_closed_forms():
    rng = np.random.default_rng(15)
    G1 = rng.standard_normal((18, 25))
    G2 = rng.standard_normal((18, 25))
    beta = 0.9
    M1 = osp.ema(np.zeros((18, 25)), G1, beta)
    assert np.allclose(M1, 0.1 * G1, atol=1e-15)
    # s(M) = (1 - beta) s(G) after one arrival from zero
    assert np.allclose(np.linalg.svd(M1, compute_uv=False), 0.1 * np.linalg.svd(G1, compute_uv=False))
    M2 = osp.ema(M1, G2, beta)
    assert np.allclose(M2, beta * 0.1 * G1 + 0.1 * G2, atol=1e-15)
    # a repeated arrival of the same gradient converges geometrically to it
    M = np.zeros_like(G1)
    for k in range(1, 6):
        M = osp.ema(M, G1, beta)
        assert np.allclose(M, (1 - beta ** k) * G1, atol=1e-14)


def test_alignment_of_rotated_subspace_is_cos_squared():
    # workload generator check: exp(eps A) rotates every principal angle by eps
    g = torch.Generator().manual_seed(0)
    Q = workloads.orthonormal(80, 6, g, "cpu")
    for eps in (0.0, 0.05, 0.2):
        Q2 = workloads.rotate_columns(Q, eps, g)
        assert torch.allclose(Q2.T @ Q2, torch.eye(6, dtype=torch.float64), atol=1e-12)
        ov = float(torch.linalg.norm(Q.T @ Q2) ** 2)
        assert abs(ov - 6 * np.cos(eps) ** 2) < 1e-10
    # eta_r for g = U V^T-aligned gradient is 1, for the orthogonal complement 0
    U, s, V = _basis(20, 14, 3, 21)
    g_in = U @ np.diag([3.0, 2.0, 1.0]) @ V.T
    assert abs(osp.alignment(g_in, U, V) - 1.0) < 1e-12


def test_planted_mistakes_are_caught_by_the_pins(monkeypatch):
    """Each mutation of the oracle's arithmetic must fail at least one pin."""
    M, U, s, V = _closed_form_case()
    alpha, tau = 0.3, 1.0

    def closed_form_ok():
        Uo, so, Vo = osp.top_r_svd(M, 6)
        do = osp.filter_weights(so, tau)
        got = osp.correct(M, Uo, do, Vo, alpha)
        d_true = s / (s + tau)
        expect = (U * ((alpha + (1 - alpha) * d_true ** 2) * s)) @ V.T
        return np.allclose(got, expect, atol=1e-10)

    def lemma1_ok():
        # the tight case: a gradient inside the prior's subspaces
        G = (U * np.arange(1.0, 7.0)) @ V.T
        d = osp.filter_weights(s, tau)
        return np.linalg.norm(osp.two_sided_filter(G, U, d, V)) <= np.linalg.norm(G) * (1 + 1e-12)

    assert closed_form_ok() and lemma1_ok()
    orig_tsf = osp.two_sided_filter
    orig_fw = osp.filter_weights
    mutants = {
        "one-sided filter": lambda G, U_, d, V_: U_ @ (d[:, None] * (U_.T @ G @ V_)) @ V_.T,
        "no filter": lambda G, U_, d, V_: U_ @ (U_.T @ G @ V_) @ V_.T,
        "sign flip": lambda G, U_, d, V_: -orig_tsf(G, U_, d, V_),
        "filter squared twice": lambda G, U_, d, V_: orig_tsf(G, U_, d ** 2, V_),
    }
    for name, fn in mutants.items():
        monkeypatch.setattr(osp, "two_sided_filter", fn)
        assert not closed_form_ok(), name
        monkeypatch.setattr(osp, "two_sided_filter", orig_tsf)
    for name, fn in {"tau/(s+tau)": lambda s_, t: t / (s_ + t),
                     "s/(s-tau)": lambda s_, t: s_ / (s_ - t)}.items():
        monkeypatch.setattr(osp, "filter_weights", fn)
        assert not closed_form_ok(), name
        monkeypatch.setattr(osp, "filter_weights", orig_fw)
    # swapped blend weights
    orig_correct = osp.correct
    monkeypatch.setattr(osp, "correct",
                        lambda G, U_, d, V_, a: (1 - a) * np.asarray(G) + a * orig_tsf(G, U_, d, V_))
    assert not closed_form_ok()
    monkeypatch.setattr(osp, "correct", orig_correct)
    # amplifying filter weights break Lemma 1
    monkeypatch.setattr(osp, "filter_weights", lambda s_, t: 1.0 + s_ / (s_ + t))
    assert not lemma1_ok()


def test_correct_rows_equals_the_rows_of_the_whole_correction():
    """The row-sampled correction (for matrices too large to form whole)
    gives exactly the rows of the whole correction, whether G is an array or
    a row-block callable, including a block boundary at 1024 rows."""
    rng = np.random.default_rng(5)
    m, n, r = 2100, 70, 6
    G = rng.standard_normal((m, n))
    U = np.linalg.qr(rng.standard_normal((m, r)))[0]
    V = np.linalg.qr(rng.standard_normal((n, r)))[0]
    d = rng.uniform(0.2, 0.9, r)
    rows = np.array([0, 1023, 1024, 2099, 17])
    whole = osp.correct(G, U, d, V, 0.3)
    got = osp.correct_rows(G, U, d, V, 0.3, rows)
    assert np.allclose(got, whole[rows], rtol=1e-12, atol=1e-12)
    got2 = osp.correct_rows(lambda a, b: G[a:b], U, d, V, 0.3, rows)
    assert np.allclose(got2, whole[rows], rtol=1e-12, atol=1e-12)


def _orthonormal_columns(rows, cols, seed):
    q, r = np.linalg.qr(np.random.default_rng(seed).standard_normal((rows, cols)))
    return q * np.sign(np.diag(r))


def test_projector_distance_is_the_sine_of_the_principal_angles():
    """||P1 - P2||_F^2 = 2 sum_i sin^2(theta_i) for r-dimensional subspaces at
    principal angles theta_i, so the distance over sqrt(2 r) is sin(eps) when
    every angle is eps, 1 for orthogonal subspaces and 0 for a rotation of the
    basis inside its span (the diagnostic the parity tests report)."""
    for m, method in ((50, "projector"), (50, "residual"), (5000, "auto")):
        r = 4
        B = _orthonormal_columns(m, 2 * r, 31)
        Q, W = B[:, :r], B[:, r:]
        dist = lambda A, C: osp.projector_distance(A, C, method=method)
        for eps in (0.0, 0.05, 0.2, 0.7, np.pi / 2):
            Q2 = Q * np.cos(eps) + W * np.sin(eps)
            assert abs(dist(Q, Q2) - np.sin(eps)) < 1e-13, (m, method, eps)
        assert abs(dist(Q, W) - 1.0) < 1e-13
        R = _orthonormal_columns(r, r, 32)
        assert dist(Q, Q @ R) < 1e-13
        # unequal angles a, b on two of the columns (the other two shared)
        a, b = 0.3, 1.1
        Q3 = Q.copy()
        Q3[:, 0] = Q[:, 0] * np.cos(a) + W[:, 0] * np.sin(a)
        Q3[:, 1] = Q[:, 1] * np.cos(b) + W[:, 1] * np.sin(b)
        expect = np.sqrt((np.sin(a) ** 2 + np.sin(b) ** 2) / r)
        assert abs(dist(Q, Q3) - expect) < 1e-13


def test_rel_fro_on_hand_computed_pairs():
    """||a - b||_F / ||b||_F: the reference b is the denominator."""
    a = np.array([[1.0, 0.0], [0.0, 0.0]])
    b = np.array([[0.0, 2.0], [0.0, 0.0]])
    assert abs(osp.rel_fro(a, b) - np.sqrt(5.0) / 2.0) < 1e-15      # ||b|| = 2, ||a|| = 1
    assert abs(osp.rel_fro(b, a) - np.sqrt(5.0)) < 1e-15
    c = np.array([3.0, 4.0])
    assert abs(osp.rel_fro(1.1 * c, c) - 0.1) < 1e-14                # a relative scale error
    assert osp.rel_fro(c, c) == 0.0
    assert osp.rel_fro(c, np.zeros(2)) == 5.0                        # zero reference: absolute error


def test_alignment_splits_a_gradient_into_its_in_and_out_of_subspace_energy():
    """eta_r = ||U^T g V||^2 / ||g||^2 (App. G): for g = U C V^T + g_out with
    U^T g_out V = 0, eta = ||C||^2 / (||C||^2 + ||g_out||^2)."""
    m, n, r = 30, 22, 3
    U = _orthonormal_columns(m, r, 41)
    V = _orthonormal_columns(n, r, 42)
    C = np.array([[2.0, 0.5, 0.0], [0.0, 1.0, -1.0], [0.25, 0.0, 3.0]])
    g_in = U @ C @ V.T
    N = np.random.default_rng(43).standard_normal((m, n))
    g_out = N - U @ (U.T @ N)                    # U^T g_out = 0
    for scale in (0.5, 1.0, 3.0):
        g = g_in + scale * g_out
        a = np.sum(C ** 2)
        b = scale ** 2 * np.sum(g_out ** 2)
        assert abs(osp.alignment(g, U, V) - a / (a + b)) < 1e-13, scale
    assert abs(osp.alignment(g_in, U, V) - 1.0) < 1e-13
    assert osp.alignment(g_out, U, V) < 1e-28
    assert osp.alignment(np.zeros((m, n)), U, V) == 0.0


def test_planted_mistakes_in_the_comparison_helpers_are_caught(monkeypatch):
    """Plausible slips in the helpers that gate every parity assertion each
    fail one of the pins above."""
    mutants = {
        "projector_distance": [
            lambda U1, U2, method="auto": 0.0,
            lambda U1, U2, method="auto": float(np.linalg.norm(U1 @ U1.T - U2 @ U2.T)),
            lambda U1, U2, method="auto": float(np.linalg.norm(U1 @ U1.T - U2 @ U2.T) / np.sqrt(U1.shape[1])),
            lambda U1, U2, method="auto": float(np.linalg.norm(U1 - U2) / np.sqrt(2.0 * U1.shape[1])),
            lambda U1, U2, method="auto": float(np.linalg.norm(U1 - U2 @ (U2.T @ U1)) / np.sqrt(2.0 * U1.shape[1])),
        ],
        "rel_fro": [
            lambda a, b: float(np.linalg.norm(np.subtract(a, b)) / np.linalg.norm(a)),
            lambda a, b: float(np.linalg.norm(np.subtract(a, b))),
            lambda a, b: float(np.linalg.norm(np.subtract(a, b)) ** 2 / np.linalg.norm(b) ** 2),
        ],
        "alignment": [
            lambda g, U, V: float(np.linalg.norm(U.T @ g @ V) / np.linalg.norm(g)),
            lambda g, U, V: float(np.linalg.norm(U.T @ g) ** 2 / np.linalg.norm(g) ** 2),
            lambda g, U, V: float(np.linalg.norm(U.T @ g @ V) ** 2),
        ],
    }
    pins = {
        "projector_distance": test_projector_distance_is_the_sine_of_the_principal_angles,
        "rel_fro": test_rel_fro_on_hand_computed_pairs,
        "alignment": test_alignment_splits_a_gradient_into_its_in_and_out_of_subspace_energy,
    }
    for name, fns in mutants.items():
        orig = getattr(osp, name)
        for k, fn in enumerate(fns):
            monkeypatch.setattr(osp, name, fn)
            with pytest.raises(AssertionError), np.errstate(all="ignore"):
                pins[name]()
            monkeypatch.setattr(osp, name, orig)
        pins[name]()


def test_transposed_filter_operand_is_caught_by_idempotence():
    """A transposed inner operand (U X^T V^T in place of U X V^T, which the
    closed form cannot see because X is diagonal there) breaks the projector
    identity at tau = 0."""
    U, s, V = _basis(26, 19, 5, 4)
    d = osp.filter_weights(s, 0.0)
    A = np.random.default_rng(5).standard_normal((26, 19))

    def transposed(G, U_, d_, V_):
        X = U_.T @ np.asarray(G, dtype=np.float64) @ V_
        Xf = d_[:, None] * X.T * d_[None, :]
        return U_ @ Xf @ V_.T

    P = lambda X: transposed(X, U, d, V)
    assert not np.allclose(P(P(A)), P(A), atol=1e-12)
    Q = lambda X: osp.two_sided_filter(X, U, d, V)
    assert np.allclose(Q(Q(A)), Q(A), atol=1e-12)


@pytest.mark.parametrize("m,n,r", [(60, 90, 7), (90, 60, 7), (50, 50, 50), (33, 80, 1)])
def test_gram_route_gives_the_svd_triplets(m, n, r):
    """The Gram route to the top-r triplets against LAPACK's SVD (a different
    routine): singular values, projectors, and the triplet relations
    M v = s u, M^T u = s v, on a spectrum with distinct values."""
    rng = np.random.default_rng(m + 3 * n + r)
    U, s, V = _basis(m, n, min(m, n), m * n)
    s = np.geomspace(50.0, 0.5, min(m, n))
    M = (U * s) @ V.T + 1e-3 * rng.standard_normal((m, n))
    Ug, sg, Vg = osp.top_r_svd_gram(M, r)
    Uo, so, Vo = osp.top_r_svd(M, r)
    assert np.allclose(sg, so, rtol=1e-10, atol=1e-12 * so[0])
    assert np.all(np.diff(sg) <= 0)
    assert osp.projector_distance(Ug, Uo) < 1e-9
    assert osp.projector_distance(Vg, Vo) < 1e-9
    assert np.allclose(M @ Vg, Ug * sg, atol=1e-9 * so[0])
    assert np.allclose(M.T @ Ug, Vg * sg, atol=1e-9 * so[0])
    assert np.allclose(Ug.T @ Ug, np.eye(r), atol=1e-9)
    assert np.allclose(Vg.T @ Vg, np.eye(r), atol=1e-9)


def test_gram_route_on_a_rank_deficient_matrix():
    """Rank 3 asked for r = 5: the constructed values, then zeros with zero
    columns on the derived side (the filter then gives d = 0 there)."""
    M, U, s, V = _closed_form_case(40, 28, 3, 8)
    Ug, sg, Vg = osp.top_r_svd_gram(M, 5)
    assert np.allclose(sg[:3], s, rtol=1e-12)
    assert np.all(sg[3:] < 1e-6)
    assert osp.projector_distance(Ug[:, :3], U) < 1e-10
    assert osp.projector_distance(Vg[:, :3], V) < 1e-6
    d = osp.filter_weights(np.where(sg < 1e-6, 0.0, sg), 1e-3)
    assert np.all(d[3:] == 0)
