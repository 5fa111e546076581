"""Pins of the corrected-AdamW oracle (paper Alg. 1; App. I optimiser).

The oracle is checked against other implementations and closed forms:
torch.optim.AdamW and torch.nn.utils.clip_grad_norm_ in float64 on the CPU
(independent library routines), the closed form of the first step from zero
moments, the clipping invariants, and the norm identity the library uses to
clip without a pass over G_proj.  The last test plants plausible mistakes into
a copy of the oracle and checks that these pins catch each of them.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import adamw as oad
from oracle import spectral as osp

HP = dict(lr=2e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)


def _state(shape, seed):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal(shape)
    m = 1e-3 * rng.standard_normal(shape)
    v = 1e-6 * rng.random(shape) + 1e-8
    return W, m, v


@pytest.mark.parametrize("wd", [0.0, 0.01, 0.1])
def test_matches_torch_adamw_over_several_steps(wd):
    shape = (7, 5)
    W, m, v = _state(shape, 1)
    rng = np.random.default_rng(2)
    grads = [1e-3 * rng.standard_normal(shape) for _ in range(6)]
    p = torch.nn.Parameter(torch.tensor(W, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=1e-2, betas=(0.9, 0.999), eps=1e-8, weight_decay=wd)
    Wo, mo, vo = W.copy(), np.zeros(shape), np.zeros(shape)
    for t, g in enumerate(grads, start=1):
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        Wo, mo, vo = oad.adamw(Wo, mo, vo, g, 1e-2, 0.9, 0.999, 1e-8, wd, t)
    st = opt.state[p]
    assert np.allclose(Wo, p.detach().numpy(), rtol=1e-13, atol=1e-15)
    assert np.allclose(mo, st["exp_avg"].numpy(), rtol=1e-13, atol=1e-20)
    assert np.allclose(vo, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=1e-24)


def test_first_step_from_zero_moments_is_a_signed_unit_step():
    # t = 1, m = v = 0: m_hat = g, v_hat = g^2, so the Adam step is g / (|g| + eps)
    W, _, _ = _state((6, 4), 3)
    g = np.random.default_rng(4).standard_normal((6, 4))
    lr, wd, eps = 0.5, 0.1, 1e-8
    Wn, mn, vn = oad.adamw(W, np.zeros_like(W), np.zeros_like(W), g, lr, 0.9, 0.999, eps, wd, 1)
    assert np.allclose(Wn, W * (1 - lr * wd) - lr * g / (np.abs(g) + eps), rtol=1e-14, atol=1e-15)
    assert np.allclose(mn, 0.1 * g, rtol=1e-15) and np.allclose(vn, 0.001 * g * g, rtol=1e-15)


@pytest.mark.parametrize("max_norm", [0.2, 1e3])
def test_clipping_matches_torch_clip_grad_norm(max_norm):
    rng = np.random.default_rng(5)
    grads = [rng.standard_normal((4, 3)), rng.standard_normal((2, 6)), rng.standard_normal((5, 5))]
    ps = [torch.nn.Parameter(torch.zeros(g.shape, dtype=torch.float64)) for g in grads]
    for p, g in zip(ps, grads):
        p.grad = torch.tensor(g, dtype=torch.float64)
    total = torch.nn.utils.clip_grad_norm_(ps, max_norm)
    N = oad.global_norm(grads)
    c = oad.clip_coefficient(N, max_norm)
    assert abs(N - float(total)) <= 1e-13 * N
    for p, g in zip(ps, grads):
        assert np.allclose(c * g, p.grad.numpy(), rtol=1e-14, atol=0)
    # the clipped norm is min(N, max_norm) up to the guard
    assert abs(oad.global_norm([c * g for g in grads]) - min(N, max_norm)) <= 1e-5 * min(N, max_norm)
    assert oad.clip_coefficient(N, 0.0) == 1.0


def test_norm_identity_used_by_the_library():
    # ||alpha G + (1-alpha) U X_f V^T||^2
    #   = alpha^2 ||G||^2 + 2 alpha (1-alpha) <X, X_f> + (1-alpha)^2 ||X_f||^2
    # for orthonormal U, V, with X = U^T G V and X_f = d X d
    U, s, V = workloads.random_orthonormal_basis(40, 30, 6, 7)
    U, V = U.numpy(), V.numpy()
    d = osp.filter_weights(s.numpy(), 0.5)
    G = np.random.default_rng(8).standard_normal((40, 30))
    alpha = 0.3
    X = U.T @ G @ V
    Xf = d[:, None] * X * d[None, :]
    lhs = np.sum(osp.correct(G, U, d, V, alpha) ** 2)
    rhs = alpha ** 2 * np.sum(G ** 2) + 2 * alpha * (1 - alpha) * np.sum(X * Xf) + (1 - alpha) ** 2 * np.sum(Xf ** 2)
    assert abs(lhs - rhs) <= 1e-12 * lhs


def test_corrected_adamw_composes_correction_clip_and_update():
    U, s, V = workloads.random_orthonormal_basis(12, 9, 3, 9)
    U, V = U.numpy(), V.numpy()
    d = osp.filter_weights(s.numpy(), 1e-3)
    rng = np.random.default_rng(10)
    mats = []
    for i in range(2):
        W, m, v = _state((12, 9), 11 + i)
        mats.append(dict(G=rng.standard_normal((12, 9)), U=U, d=d, V=V, W=W, m=m, v=v))
    out, N = oad.corrected_adamw(mats, 0.3, t=4, max_norm=0.2, **HP)
    gp = [osp.correct(x["G"], U, d, V, 0.3) for x in mats]
    assert abs(N - np.sqrt(sum(np.sum(g * g) for g in gp))) <= 1e-12 * N
    c = 0.2 / (N + 1e-6)
    for x, g, (W, m, v) in zip(mats, gp, out):
        Wr, mr, vr = oad.adamw(x["W"], x["m"], x["v"], c * g, t=4, **HP)
        assert np.array_equal(W, Wr) and np.array_equal(m, mr) and np.array_equal(v, vr)


def test_planted_mistakes_are_caught():
    """Each variant below is a plausible slip in writing AdamW; a pin above
    (re-run here on the variant) must reject it."""
    shape = (5, 4)
    W, _, _ = _state(shape, 12)
    rng = np.random.default_rng(13)
    grads = [1e-3 * rng.standard_normal(shape) for _ in range(4)]

    def torch_run(wd):
        p = torch.nn.Parameter(torch.tensor(W, dtype=torch.float64))
        opt = torch.optim.AdamW([p], lr=1e-2, betas=(0.9, 0.999), eps=1e-8, weight_decay=wd)
        for g in grads:
            p.grad = torch.tensor(g, dtype=torch.float64)
            opt.step()
        return p.detach().numpy()

    def no_bias_correction(W, m, v, g, lr, b1, b2, eps, wd, t):
        W = W * (1 - lr * wd)
        m = b1 * m + (1 - b1) * g
        v = b2 * v + (1 - b2) * g * g
        return W - lr * m / (np.sqrt(v) + eps), m, v

    def coupled_decay(W, m, v, g, lr, b1, b2, eps, wd, t):   # Adam with L2, not AdamW
        return oad.adamw(W, m, v, g + wd * W, lr, b1, b2, eps, 0.0, t)

    def eps_inside_sqrt(W, m, v, g, lr, b1, b2, eps, wd, t):
        W = W * (1 - lr * wd)
        m = b1 * m + (1 - b1) * g
        v = b2 * v + (1 - b2) * g * g
        return W - lr * (m / (1 - b1 ** t)) / np.sqrt(v / (1 - b2 ** t) + eps), m, v

    ref = torch_run(0.1)
    for bad in (no_bias_correction, coupled_decay, eps_inside_sqrt):
        Wb, mb, vb = W.copy(), np.zeros(shape), np.zeros(shape)
        for t, g in enumerate(grads, start=1):
            Wb, mb, vb = bad(Wb, mb, vb, g, 1e-2, 0.9, 0.999, 1e-8, 0.1, t)
        assert not np.allclose(Wb, ref, rtol=1e-13, atol=1e-15), bad.__name__
    # clipping each matrix by its own norm instead of the global one
    big = [np.full((2, 2), 3.0), np.full((2, 2), 0.1)]
    per_matrix = [g * oad.clip_coefficient(oad.global_norm([g]), 1.0) for g in big]
    glob = [g * oad.clip_coefficient(oad.global_norm(big), 1.0) for g in big]
    assert not np.allclose(per_matrix[1], glob[1])
