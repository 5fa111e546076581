"""GPU parity of the corrected AdamW step (Alg. 1 update; App. I optimiser)
against the CPU oracle.

Both sides get the same prior (U, d, V) and the same fp32 optimiser state;
the oracle forms G_proj, the global norm, the clip and the AdamW step in
float64.  Compared: the weight update W_new - W_old, the moments and the
reported norm, by relative Frobenius error: 1e-4 for fp32 gradients, 2e-2
for bf16 gradients (fp32 accumulation), as for the correction itself.  The
cases cover every kernel path: fp32 (64 x 64 tiles), bf16 with a padded rank
the streamed-tile kernel does not take, the streamed-tile kernel with 16-byte
and with only 4-byte aligned state, more than 16 matrices in one call (the
norm accumulated over launches), and a full-size 70B-class layer on sampled
rows.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import adamw as oad
from oracle import spectral as osp

pytestmark = pytest.mark.gpu

# lr large enough that the update (~1e-3 here) dominates fp32's rounding of
# W itself (half an ulp, ~1e-7 for |W| ~ 1), which no implementation avoids
HP = dict(lr=0.1, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)


@pytest.fixture(scope="module")
def pk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_14339_amd as pk
    return pk


def _case(m, n, r, seed, dtype, t):
    """Gradient, an orthonormal prior with soft weights, and an optimiser state."""
    G = workloads.gaussian((m, n), seed=seed, dtype=dtype)
    U, s, V = workloads.random_orthonormal_basis(m, n, r, seed + 1)
    d = osp.filter_weights(s.numpy(), 0.3)
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((m, n)).astype(np.float32)
    if t == 1:
        m1 = np.zeros((m, n), np.float32)
        m2 = np.zeros((m, n), np.float32)
    else:
        m1 = (0.05 * rng.standard_normal((m, n))).astype(np.float32)
        m2 = (rng.random((m, n)) + 0.5).astype(np.float32)
    return dict(G=G, U=U.float(), d=torch.tensor(d, dtype=torch.float32), V=V.float(), W=W, m1=m1, m2=m2)


def _run(pk, cases, r, alpha, t, max_norm, dtype, misalign=False):
    dev = torch.device("cuda")
    items, states = [], []
    for c in cases:
        m, n = c["G"].shape
        st = []
        for a in (c["W"], c["m1"], c["m2"]):
            if misalign:    # 4-byte aligned views, not 16-byte aligned
                buf = torch.empty(a.size + 1, dtype=torch.float32, device=dev)
                v = buf[1:].view(m, n)
                v.copy_(torch.from_numpy(a))
            else:
                v = torch.from_numpy(a).to(dev)
            st.append(v)
        states.append(st)
        items.append(dict(G=c["G"].to(dev), prior=(c["U"].to(dev), c["d"].to(dev), c["V"].to(dev)),
                          ws=pk.workspace(m, n, r, 0, dtype, dev), state=tuple(st)))
    norm = torch.zeros(1, device=dev)
    pk.sc_correct_adamw_batched(items, r, alpha, step=t, max_norm=max_norm, dtype=dtype, norm_out=norm, **HP)
    torch.cuda.synchronize()
    return [tuple(x.double().cpu().numpy() for x in st) for st in states], float(norm.item())


def _oracle(cases, alpha, t, max_norm):
    mats = [dict(G=c["G"].double().numpy(), U=c["U"].double().numpy(), d=c["d"].double().numpy(),
                 V=c["V"].double().numpy(), W=c["W"], m=c["m1"], v=c["m2"]) for c in cases]
    return oad.corrected_adamw(mats, alpha, t=t, max_norm=max_norm, **HP)


def _compare(cases, got, ref, tol):
    for c, (Wg, mg, vg), (Wo, mo, vo) in zip(cases, got, ref):
        W0 = c["W"].astype(np.float64)
        assert osp.rel_fro(Wg - W0, Wo - W0) <= tol, "weight update differs"
        assert osp.rel_fro(mg, mo) <= tol, "first moment differs"
        assert osp.rel_fro(vg, vo) <= tol, "second moment differs"


@pytest.mark.parametrize("t", [1, 5])
@pytest.mark.parametrize("max_norm", [0.0, 1.0])
def test_fp32_matches_oracle(pk, t, max_norm):
    cases = [_case(256, 256, 8, 3, torch.float32, t), _case(130, 70, 8, 4, torch.float32, t)]
    got, N = _run(pk, cases, 8, 0.3, t, max_norm, torch.float32)
    ref, No = _oracle(cases, 0.3, t, max_norm)
    assert abs(N - No) <= 1e-5 * No
    if max_norm > 0:
        assert No > max_norm          # clipping is active in this case
    _compare(cases, got, ref, 1e-4)


@pytest.mark.parametrize("m,n,r", [(300, 200, 7), (129, 4104, 40), (1000, 17, 3)])
def test_bf16_padded_ranks_off_the_tile_kernel(pk, m, n, r):
    # padded ranks 32 and 64 / unaligned rows: the 128 x 128 tile kernel
    cases = [_case(m, n, r, 10 + r, torch.bfloat16, 5)]
    got, N = _run(pk, cases, r, 0.3, 5, 0.5, torch.bfloat16)
    ref, No = _oracle(cases, 0.3, 5, 0.5)
    assert abs(N - No) <= 5e-3 * No
    _compare(cases, got, ref, 2e-2)


@pytest.mark.parametrize("misalign", [False, True])
@pytest.mark.parametrize("m,n,r", [(512, 384, 64), (256, 1024, 128), (400, 264, 150)])
def test_bf16_streamed_tile_kernel(pk, m, n, r, misalign):
    # padded ranks 64, 128, 192; 16-byte or only 4-byte aligned state
    cases = [_case(m, n, r, 20 + r, torch.bfloat16, 5), _case(m // 2, n, r, 21 + r, torch.bfloat16, 5)]
    got, N = _run(pk, cases, r, 0.3, 5, 2.0, torch.bfloat16, misalign=misalign)
    ref, No = _oracle(cases, 0.3, 5, 2.0)
    assert abs(N - No) <= 5e-3 * No
    _compare(cases, got, ref, 2e-2)


def test_norm_spans_more_than_one_launch(pk):
    # 18 matrices: two launches of the norm kernel accumulate one global norm
    cases = [_case(64 + 8 * i, 96, 8, 40 + i, torch.bfloat16, 3) for i in range(18)]
    got, N = _run(pk, cases, 8, 0.3, 3, 1.0, torch.bfloat16)
    ref, No = _oracle(cases, 0.3, 3, 1.0)
    assert No > 1.0
    assert abs(N - No) <= 5e-3 * No
    _compare(cases, got, ref, 2e-2)


def test_deterministic_and_no_side_effects_on_error(pk):
    cases = [_case(256, 512, 64, 60, torch.bfloat16, 5)]
    a, Na = _run(pk, cases, 64, 0.3, 5, 1.0, torch.bfloat16)
    b, Nb = _run(pk, cases, 64, 0.3, 5, 1.0, torch.bfloat16)
    assert Na == Nb
    for x, y in zip(a[0], b[0]):
        assert np.array_equal(x, y)
    # a bad hyperparameter is rejected before anything is enqueued
    dev = torch.device("cuda")
    c = cases[0]
    W = torch.from_numpy(c["W"]).to(dev)
    m1, m2 = torch.zeros_like(W), torch.zeros_like(W)
    item = dict(G=c["G"].to(dev), prior=(c["U"].to(dev), c["d"].to(dev), c["V"].to(dev)),
                ws=pk.workspace(256, 512, 64, 0, torch.bfloat16, dev), state=(W, m1, m2))
    with pytest.raises(pk.AcscError) as e:
        pk.sc_correct_adamw_batched([item], 64, 0.3, lr=1e-2, beta1=1.0, step=1)
    assert e.value.code == pk.ACSC_EINVAL
    with pytest.raises(pk.AcscError):
        pk.sc_correct_adamw_batched([item], 64, 0.3, lr=1e-2, step=0)
    torch.cuda.synchronize()
    assert torch.equal(W.cpu(), torch.from_numpy(c["W"])) and not m1.any() and not m2.any()


def test_70b_class_layer_full_size_sampled_rows(pk):
    """The three matrices of one 70B-class layer (8192 x 8192, 8192 x 28672,
    28672 x 8192, bf16, r = 128) at full size in one call: the norm against
    the oracle's exact G_proj norm (formed in row blocks), the update on
    sampled rows."""
    cfg = workloads.CONFIGS[5]
    gs = cfg.grad
    r = gs.r[0]
    dev = torch.device("cuda")
    items, host = [], []
    for j, (m, n) in enumerate(gs.shapes):
        G_anc, G = workloads.grad_pair_fast(gs, 5, 0, j, dev)
        M = torch.zeros(m, n, device=dev)
        U, s, V, d = pk.sc_build_prior(G_anc, M, r, workloads.BETA, workloads.TAU, cfg.oversample,
                                       cfg.power_iters, seed=7, dtype=torch.bfloat16)
        del M, G_anc
        gen = torch.Generator(device=dev).manual_seed(100 + j)
        W = torch.randn(m, n, device=dev, generator=gen)
        m1 = 1e-4 * torch.randn(m, n, device=dev, generator=gen)
        m2 = 1e-8 * (torch.rand(m, n, device=dev, generator=gen) + 0.5)
        rows = np.r_[0:16, m // 2:m // 2 + 16, m - 16:m]
        host.append(dict(G=G, U=U.double().cpu().numpy(), d=d.double().cpu().numpy(),
                         V=V.double().cpu().numpy(), rows=rows, W=W[rows].double().cpu().numpy(),
                         m=m1[rows].double().cpu().numpy(), v=m2[rows].double().cpu().numpy()))
        items.append(dict(G=G, prior=(U, d, V), ws=pk.workspace(m, n, r, 0, torch.bfloat16, dev),
                          state=(W, m1, m2)))
    norm = torch.zeros(1, device=dev)
    hp = dict(lr=2e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
    pk.sc_correct_adamw_batched(items, r, workloads.ALPHA, step=3, max_norm=0.2, norm_out=norm, **hp)
    torch.cuda.synchronize()
    # oracle: exact global norm of the G_proj (row blocks), then sampled rows of the step
    sq = 0.0
    sampled = []
    for h in host:
        G, U, d, V = h["G"], h["U"], h["d"], h["V"]
        m = U.shape[0]
        get = lambda a, b: G[a:b].double().cpu().numpy()
        X = np.zeros((U.shape[1], V.shape[1]))
        for a in range(0, m, 2048):
            X += U[a:a + 2048].T @ (get(a, a + 2048) @ V)
        Xf = d[:, None] * X * d[None, :]
        FV = Xf @ V.T
        for a in range(0, m, 2048):
            gp = workloads.ALPHA * get(a, a + 2048) + (1 - workloads.ALPHA) * (U[a:a + 2048] @ FV)
            sq += float(np.sum(gp * gp))
        sampled.append(osp.correct_rows(get, U, d, V, workloads.ALPHA, h["rows"]))
    No = np.sqrt(sq)
    assert abs(norm.item() - No) <= 5e-3 * No
    c = oad.clip_coefficient(No, 0.2)
    assert c < 1.0
    for h, gp, it in zip(host, sampled, items):
        Wo, mo, vo = oad.adamw(h["W"], h["m"], h["v"], c * gp, t=3, **hp)
        W, m1, m2 = (x[h["rows"]].double().cpu().numpy() for x in it["state"])
        assert osp.rel_fro(W - h["W"], Wo - h["W"]) <= 2e-2
        assert osp.rel_fro(m1, mo) <= 2e-2 and osp.rel_fro(m2, vo) <= 2e-2
