"""GPU parity of the spectral corrector at the larger workload shapes (Sec. 3.2;
Alg. 1; App. E): every 8B-class matrix against the whole oracle, the
anchor-staleness sweep on every 8B-class shape (one prior against rotated
masked gradients; three anchor arrivals, rebuilt cold and warm-started), and
the 70B-class four-layer step (the batch the benchmark times, which takes the
fused EMA pass), whose priors are compared with the oracle's own SVD and whose
corrected gradients are compared on sampled rows.

Tolerance of the corrected gradient against the float64 oracle: 2e-2
relative Frobenius error (bf16 inputs, fp32 accumulation).  The oracle's
top-r SVD of matrices wider than 4096 goes through the Gram matrix of the
shorter side (the same triplets; a full LAPACK SVD there takes minutes).
"""
import functools
import time

import numpy as np
import pytest
import torch

import workloads
from oracle import spectral as osp

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2


def _oracle_svd(M, r):
    return osp.top_r_svd_gram(M, r) if max(M.shape) > 4096 else osp.top_r_svd(M, r)


def _prior_vs_oracle(U, s, V, Uo, so, Vo, lead_tol=1e-3):
    """The unique parts of a prior against the oracle's: singular values (the
    leading half tight, the rest within the bf16 bound, since subspace
    iteration converges on sigma_j at (sigma_{k+1} / sigma_j)^(2q+1)) and the
    left and right projectors."""
    r = s.shape[0]
    rel = np.abs(s - so) / so
    assert np.max(rel[: max(r // 2, 1)]) < lead_tol, np.max(rel[: max(r // 2, 1)])
    assert np.max(rel) < TOL_BF16, np.max(rel)
    assert osp.projector_distance(U, Uo) < TOL_BF16
    assert osp.projector_distance(V, Vo) < TOL_BF16


@pytest.fixture(scope="module")
def pk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_14339_amd as pk
    return pk


def _np(t):
    return t.detach().double().cpu().numpy()


def _build_and_correct(pk, G_anc, G_mask, r, p, q, seed):
    m, n = G_anc.shape
    M = torch.zeros(m, n, device="cuda")
    U, s, V, d = pk.sc_build_prior(G_anc.cuda(), M, r, workloads.BETA, workloads.TAU, p, q, seed=seed)
    out = pk.sc_correct(G_mask.cuda(), U, d, V, workloads.ALPHA)
    torch.cuda.synchronize()
    return M, U, s, V, d, out


@pytest.mark.parametrize("mat", [1, 0, 2, 3])
def test_8b_class_build_and_correct_match_oracle(pk, mat):
    """C3: the 4096 x 1024 (GQA k/v), 4096 x 4096 and the 4096 x 14336 /
    14336 x 4096 MLP gradients, rank-64 signal, r = 64: the EMA exactly, the
    singular values, projectors and the corrected gradient to the bf16
    bounds, all against the oracle's own prior."""
    cfg = workloads.CONFIGS[3]
    r = cfg.grad.r[0]
    gp = workloads.grad_pair(cfg.grad, 3, 0, mat, "cpu")
    M, U, s, V, d, out = _build_and_correct(pk, gp.G_anc, gp.G_mask, r, cfg.oversample, cfg.power_iters, 31)
    Mo = osp.ema(np.zeros(gp.G_anc.shape), _np(gp.G_anc), workloads.BETA)
    Uo, so, Vo = _oracle_svd(Mo, r)
    do = osp.filter_weights(so, workloads.TAU)
    ref = osp.correct(_np(gp.G_mask), Uo, do, Vo, workloads.ALPHA)
    assert osp.rel_fro(_np(M), Mo) < 1e-6
    _prior_vs_oracle(_np(U), _np(s), _np(V), Uo, so, Vo)
    Ug, Vg = _np(U), _np(V)
    assert np.abs(Ug.T @ Ug - np.eye(r)).max() < 1e-4
    assert np.abs(Vg.T @ Vg - np.eye(r)).max() < 1e-4
    assert osp.rel_fro(_np(out), ref) <= TOL_BF16


@functools.lru_cache(maxsize=4)
def _c4_oracle(mat):
    """The oracle's top-128 SVD of the EMA of C4 matrix ``mat`` after one
    anchor arrival; truncating it gives the top-r prior for every r <= 128."""
    spec = workloads.CONFIGS[4].grad
    base = workloads.grad_pair(spec, 4, 0, mat, "cpu")
    Mo = osp.ema(np.zeros(base.G_anc.shape), _np(base.G_anc), workloads.BETA)
    Uo, so, Vo = _oracle_svd(Mo, 128)
    return base, Uo, so, Vo


@pytest.mark.parametrize("mat", [1, 0, 2, 3])
@pytest.mark.parametrize("r", [16, 64, 128])
def test_staleness_sweep_matches_oracle(pk, r, mat):
    """C4: the masked gradient's signal subspaces rotated from the anchor's by
    exp(eps A), eps in {0, 0.05, 0.2}, prior rank r in {16, 64, 128}, three
    power iterations, on every 8B-class shape.  The prior is built once from
    the anchor and reused for the three rotated gradients.

    For r up to the signal rank (64) the top-r subspace is well separated and
    the whole prior is compared with the oracle's.  At r = 128 the last 64
    directions lie in the noise bulk, whose singular values are nearly
    degenerate: those directions are not unique, so the unique part is
    compared (the signal subspace and its singular values).  The corrected
    gradients are compared with the oracle's correction under the oracle's
    own prior wherever that correction is unique: at every r up to the
    signal rank, and at r = 128 while the masked gradient's energy off the
    signal subspace is only noise (eps <= 0.05).  At r = 128 and eps = 0.2
    the rotated-out signal (sin 0.2 of it) meets the prior's 64 bulk
    directions.  Those are not resolved by the subspace iteration (bulk
    values within 2% of each other converge as 0.98^(2q+1)), so they are
    some 64 directions near the top of the bulk rather than the exact SVD's,
    and the correction moves by a few percent with them (two exact SVDs of
    M and of M perturbed at bf16 rounding agree to 0.3% there).  In that
    case the oracle's correction is taken under the GPU's prior, which
    checks the correction kernels, and the gap to the oracle's prior is
    printed: parity of the prior itself is partial there."""
    cfg = workloads.CONFIGS[4]
    spec = cfg.grad
    base, Uo_full, so_full, Vo_full = _c4_oracle(mat)
    m, n = base.G_anc.shape
    M = torch.zeros(m, n, device="cuda")
    U, s, V, d = pk.sc_build_prior(base.G_anc.cuda(), M, r, workloads.BETA, workloads.TAU, cfg.oversample,
                                   cfg.power_iters, seed=41)
    torch.cuda.synchronize()
    Uo, so, Vo = Uo_full[:, :r], so_full[:r], Vo_full[:, :r]
    do = osp.filter_weights(so, workloads.TAU)
    assert osp.rel_fro(_np(M), osp.ema(np.zeros((m, n)), _np(base.G_anc), workloads.BETA)) < 1e-6
    rank = spec.rank
    Ug, sg, Vg = _np(U), _np(s), _np(V)
    if r <= rank:
        _prior_vs_oracle(Ug, sg, Vg, Uo, so, Vo)
    else:
        # k = r + p = 144 > 128: the Rayleigh-Ritz Jacobi runs in fp32, and a
        # rotation of a column pair leaves an absolute error of ~1e-7 times the
        # larger column in the smaller one; the noise columns are 100x below
        # the leading ones, so their orthogonality holds to ~1e-3
        assert np.abs(Ug.T @ Ug - np.eye(r)).max() < 5e-3
        assert np.abs(Vg.T @ Vg - np.eye(r)).max() < 5e-3
        _prior_vs_oracle(Ug[:, :rank], sg[:rank], Vg[:, :rank], Uo[:, :rank], so[:rank], Vo[:, :rank])
    for eps in spec.rot_eps:
        gp = workloads.grad_pair(spec, 4, 0, mat, "cpu", rot_eps=eps)
        assert torch.equal(gp.G_anc, base.G_anc)
        out = pk.sc_correct(gp.G_mask.cuda(), U, d, V, workloads.ALPHA)
        torch.cuda.synchronize()
        Gm = _np(gp.G_mask)
        ref = osp.correct(Gm, Uo, do, Vo, workloads.ALPHA)
        if r <= rank or eps <= 0.05:
            assert osp.rel_fro(_np(out), ref) <= TOL_BF16, (r, eps)
        else:
            own = osp.correct(Gm, Ug, _np(d), Vg, workloads.ALPHA)
            assert osp.rel_fro(_np(out), own) <= TOL_BF16, (r, eps)
            print(f"\nC4 {m}x{n} r={r} eps={eps}: corrected gradient against the oracle's prior "
                  f"{osp.rel_fro(_np(out), ref):.2e} (bulk directions unresolved: projector distance "
                  f"{osp.projector_distance(Ug[:, rank:], Uo[:, rank:]):.2f}), against the GPU's prior "
                  f"{osp.rel_fro(_np(out), own):.2e}", flush=True)


@pytest.mark.parametrize("r,mat", [(16, 1), (64, 1), (64, 2)])
def test_staleness_three_arrivals_cold_rebuild_and_warm_start(pk, r, mat):
    """C4 over three anchor arrivals (Sec. 3.2: the prior is the EMA over
    arrivals; App. H: a new anchor gradient every few steps) whose signal
    subspaces drift 0.02 rad per arrival.  After each arrival the prior is
    rebuilt twice on the GPU from EMA states that receive the same arrivals:
    cold (random start, the configuration's three power iterations) and
    warm-started from the previous arrival's V with one power iteration.
    Both must match the oracle's prior of that arrival's EMA, and both
    corrections of the next masked gradient the oracle's correction."""
    cfg = workloads.CONFIGS[4]
    spec = cfg.grad
    m, n = spec.shapes[mat]
    p, q = cfg.oversample, cfg.power_iters
    M_cold = torch.zeros(m, n, device="cuda")
    M_warm = torch.zeros(m, n, device="cuda")
    Mo = np.zeros((m, n))
    V_prev = None
    for a in range(3):
        G_anc, G_mask = workloads.anchor_arrival(spec, 4, 0, mat, a, 0.02, "cpu")
        Ga = G_anc.cuda()
        Uc, sc, Vc, dc = pk.sc_build_prior(Ga, M_cold, r, workloads.BETA, workloads.TAU, p, q, seed=50 + a)
        Uw, sw, Vw, dw = pk.sc_build_prior(Ga, M_warm, r, workloads.BETA, workloads.TAU, p,
                                           q if V_prev is None else 1, seed=60 + a, V_warm=V_prev)
        torch.cuda.synchronize()
        assert torch.equal(M_cold, M_warm)
        Mo = osp.ema(Mo, _np(G_anc), workloads.BETA)
        assert osp.rel_fro(_np(M_cold), Mo) < 1e-6
        Uo, so, Vo = _oracle_svd(Mo, r)
        do = osp.filter_weights(so, workloads.TAU)
        ref = osp.correct(_np(G_mask), Uo, do, Vo, workloads.ALPHA)
        Gm = G_mask.cuda()
        for tag, (U, s, V, d) in (("cold", (Uc, sc, Vc, dc)), ("warm", (Uw, sw, Vw, dw))):
            _prior_vs_oracle(_np(U), _np(s), _np(V), Uo, so, Vo)
            out = pk.sc_correct(Gm, U, d, V, workloads.ALPHA)
            torch.cuda.synchronize()
            assert osp.rel_fro(_np(out), ref) <= TOL_BF16, (tag, a)
        V_prev = Vw.clone()


@pytest.fixture(scope="module")
def c5(pk):
    """C5, the benchmark's batch: four layers of 8192 x 8192, 8192 x 28672 and
    28672 x 8192 gradients (rank-128 signal), r = 128, (k, q) = (160, 2), one
    batched build (the EMA fused with the first pass) and one batched
    correction, in the launch configuration the benchmark times."""
    cfg = workloads.CONFIGS[5]
    spec = cfg.grad
    r, p, q = spec.r[0], cfg.oversample, cfg.power_iters
    items, corr, grads = [], [], []
    for layer in range(spec.layers):
        for mat, (m, n) in enumerate(spec.shapes):
            G_anc, G_mask = workloads.grad_pair_fast(spec, 5, layer, mat, "cuda")
            outs = (torch.empty(m, r, device="cuda"), torch.empty(r, device="cuda"),
                    torch.empty(n, r, device="cuda"), torch.empty(r, device="cuda"))
            items.append(dict(G_anc=G_anc, M=torch.zeros(m, n, device="cuda"), out=outs,
                              ws=pk.workspace(m, n, r, p, torch.bfloat16)))
            grads.append((layer, mat, G_anc, G_mask))
    pk.sc_build_prior_batched(items, r, workloads.BETA, workloads.TAU, p, q, seed=1000)
    for it, (layer, mat, G_anc, G_mask) in zip(items, grads):
        m, n = G_mask.shape
        U, s, V, d = it["out"]
        corr.append(dict(G=G_mask, prior=(U, d, V), out=torch.empty(m, n, dtype=torch.bfloat16, device="cuda"),
                         ws=pk.workspace(m, n, r, 0, torch.bfloat16)))
    pk.sc_correct_batched(corr, r, workloads.ALPHA)
    torch.cuda.synchronize()
    return dict(items=items, corr=corr, grads=grads, r=r)


def test_70b_class_step_on_sampled_rows(c5):
    """Every matrix of the C5 batch: the EMA (M = (1 - beta) G_anc) on sampled
    rows, an orthonormal prior whose leading singular values are those of the
    constructed signal scaled by (1 - beta), and 48 sampled rows of the
    corrected gradient against the oracle's row-sampled correction with the
    GPU's prior (the oracle's own prior is compared on three matrices below)."""
    spec = workloads.CONFIGS[5].grad
    r = c5["r"]
    s_sig = (1.0 - workloads.BETA) * workloads.log_spaced(spec.s_range[0], spec.s_range[1], spec.rank).numpy()
    rng = np.random.default_rng(5)
    for it, c, (layer, mat, G_anc, G_mask) in zip(c5["items"], c5["corr"], c5["grads"]):
        m, n = G_mask.shape
        rows = np.sort(rng.choice(m, 48, replace=False))
        idx = torch.tensor(rows, device="cuda")
        M_rows = _np(it["M"].index_select(0, idx))
        assert osp.rel_fro(M_rows, osp.ema(np.zeros((48, n)), _np(G_anc.index_select(0, idx)), workloads.BETA)) < 1e-6
        U, s, V, d = (_np(x) for x in it["out"])
        assert np.abs(U.T @ U - np.eye(r)).max() < 1e-3
        assert np.abs(V.T @ V - np.eye(r)).max() < 1e-3
        assert np.all(np.diff(s) <= 0) and s[-1] > 0
        # the noise is 5% of the signal scale: the leading values move by far
        # less than 1%
        assert np.max(np.abs(s[:32] - s_sig[:32]) / s_sig[:32]) < 1e-2
        got = _np(c["out"].index_select(0, idx))
        ref = osp.correct_rows(lambda a, b: _np(G_mask[a:b]), U, d, V, workloads.ALPHA, rows)
        assert osp.rel_fro(got, ref) <= TOL_BF16


@pytest.mark.parametrize("which", [0, 1, 11])
def test_70b_class_prior_matches_the_oracle_svd(c5, which):
    """C5 against the oracle's own prior for the 8192 x 8192 matrix of layer
    0, the 8192 x 28672 MLP matrix of layer 0 and the 28672 x 8192 MLP matrix
    of layer 3: the oracle's EMA of the same G_anc bits in float64, its top-128
    SVD and filter weights; all 128 singular values, both projectors, and 64
    sampled rows of the corrected gradient against the oracle's correction
    under the oracle's prior.  This covers the two paths only this batch
    takes: the fused split-k EMA pass and the fp32 Rayleigh-Ritz Jacobi at
    k = 160 (above 128)."""
    r = c5["r"]
    it, c = c5["items"][which], c5["corr"][which]
    layer, mat, G_anc, G_mask = c5["grads"][which]
    t0 = time.time()
    Mo = osp.ema(0.0, _np(G_anc), workloads.BETA)
    assert osp.rel_fro(_np(it["M"]), Mo) < 1e-6
    Uo, so, Vo = _oracle_svd(Mo, r)
    del Mo
    do = osp.filter_weights(so, workloads.TAU)
    t_oracle = time.time() - t0
    U, s, V, d = (_np(x) for x in it["out"])
    _prior_vs_oracle(U, s, V, Uo, so, Vo)
    assert np.max(np.abs(d - do)) < 1e-4
    m = G_mask.shape[0]
    rows = np.sort(np.random.default_rng(17 + which).choice(m, 64, replace=False))
    got = _np(c["out"].index_select(0, torch.tensor(rows, device="cuda")))
    ref = osp.correct_rows(lambda a, b: _np(G_mask[a:b]), Uo, do, Vo, workloads.ALPHA, rows)
    assert osp.rel_fro(got, ref) <= TOL_BF16
    print(f"\nC5 layer {layer} matrix {tuple(G_mask.shape)}: oracle EMA + top-{r} SVD {t_oracle:.1f} s; "
          f"max rel. error of s {np.max(np.abs(s - so) / so):.2e}; projector distances "
          f"{osp.projector_distance(U, Uo):.2e} / {osp.projector_distance(V, Vo):.2e}; "
          f"G_proj rows {osp.rel_fro(got, ref):.2e}", flush=True)
