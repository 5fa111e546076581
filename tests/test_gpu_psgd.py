"""GPU parity of the PowerSGD compressor with error feedback (the
data-parallel side the paper pairs with its method: Sec. 3.3, App. J F3)
against the CPU oracle.

Both sides get the same gradient G, memory E and previous Q; the oracle runs
the step in float64 (Gram-Schmidt, exact products).  Compared, by relative
Frobenius error (1e-4 for fp32 gradients, 2e-2 for bf16 gradients with fp32
accumulation): P before and after orthogonalisation, the new Q and the
output.  The new memory is checked bit for bit against its definition on the
GPU's own values, E' = fp32(fp32(E + G) - out), and against the oracle's
within the output's tolerance (E' - E'_oracle = out_oracle - out exactly, for
the same M).  Sizes span several tiles with ragged tails, more than sixteen
matrices per call, the fused and the unfused first pass, and one full
70B-class MLP matrix.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import powersgd as ops
from oracle import spectral as osp

pytestmark = pytest.mark.gpu

TOL = {torch.float32: 1e-4, torch.bfloat16: 2e-2}


@pytest.fixture(scope="module")
def pk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_14339_amd as pk
    return pk


def _case(m, n, r, seed, dtype, e_scale=0.1, rank=None):
    """G: a low-rank signal plus noise (or exactly rank `rank`), E: small
    memory, Q: Gaussian (host tensors)."""
    if rank is None:
        k = min(m, n, 24)
        U, s, V = workloads.random_orthonormal_basis(m, n, k, seed)
        sig = (U * torch.logspace(2, 0, k, dtype=torch.float64)) @ V.T
        G = sig + 0.05 * sig.norm() / np.sqrt(m * n) * workloads.gaussian((m, n), seed + 1).double()
    else:
        U, s, V = workloads.random_orthonormal_basis(m, n, rank, seed)
        G = (U * torch.logspace(1, 0, rank, dtype=torch.float64)) @ V.T
    G = G.to(dtype)
    E = (e_scale * G.float().std() * workloads.gaussian((m, n), seed + 2)).float()
    Q = workloads.gaussian((n, r), seed + 3)
    return dict(G=G, E=E, Q=Q)


def _items(pk, cases, r, dtype, out_is_g=False):
    dev = torch.device("cuda")
    items = []
    for c in cases:
        m, n = c["G"].shape
        G = c["G"].to(dev)
        items.append(dict(G=G, E=c["E"].to(dev), P=torch.zeros(m, r, device=dev), Q=c["Q"].to(dev),
                          out=G if out_is_g else torch.empty(m, n, dtype=dtype, device=dev),
                          ws=pk.psgd_workspace(m, n, r, dtype, dev)))
    return items


def _host(it):
    return {k: v.detach().cpu() for k, v in it.items() if k != "ws"}


def _check_step(c, got, dtype, label=""):
    """got: host tensors after the step; c: the step's inputs."""
    tol = TOL[dtype]
    od = "bf16" if dtype == torch.bfloat16 else "f32"
    o = ops.step(c["G"].double().numpy(), c["E"].double().numpy(), c["Q"].double().numpy(), od)
    assert osp.rel_fro(got["P"].double().numpy(), o["P_hat"]) <= tol, f"{label} P_hat differs"
    assert osp.rel_fro(got["Q"].double().numpy(), o["Q"]) <= tol, f"{label} Q differs"
    out = got["out"].double().numpy()
    assert osp.rel_fro(out, o["out"]) <= tol, f"{label} out differs"
    # the memory, bit for bit against its definition on the GPU's own values
    M = (c["E"] + c["G"].float())
    assert torch.equal(got["E"], M - got["out"].float()), f"{label} E != fp32(M - out)"
    err = np.linalg.norm(got["E"].double().numpy() - o["E"]) / np.linalg.norm(o["out"])
    assert err <= tol, f"{label} E differs from the oracle's by {err:.2e} of |out|"
    return o


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("m,n,r", [(256, 256, 8), (300, 200, 7), (129, 4104, 40), (1000, 17, 3),
                                   (520, 1032, 99), (384, 640, 150)])
def test_step_matches_oracle(pk, dtype, m, n, r):
    c = _case(m, n, r, m + n + r, dtype)
    items = _items(pk, [c], r, dtype)
    pk.psgd_step(items, r, dtype)
    torch.cuda.synchronize()
    _check_step(c, _host(items[0]), dtype)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_phases_equal_the_step_and_project_matches_oracle(pk, dtype):
    cases = [_case(700, 300, 12, 5, dtype), _case(300, 520, 12, 6, dtype)]
    a = _items(pk, cases, 12, dtype)
    b = _items(pk, cases, 12, dtype)
    pk.psgd_project(a, 12, dtype)
    torch.cuda.synchronize()
    for c, it in zip(cases, a):
        M, P = ops.project(c["G"].double().numpy(), c["E"].double().numpy(), c["Q"].double().numpy())
        assert osp.rel_fro(it["P"].double().cpu().numpy(), P) <= TOL[dtype]
        assert torch.equal(it["E"].cpu(), c["E"] + c["G"].float())      # M = fp32(E + G), in place
    pk.psgd_orthogonalize(a, 12, dtype)
    pk.psgd_decompress(a, 12, dtype)
    pk.psgd_step(b, 12, dtype)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        for k in ("E", "P", "Q", "out"):
            assert torch.equal(x[k], y[k]), k


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_steps_carry_memory_and_warm_start(pk, dtype):
    """Four steps on changing gradients: at every step the oracle takes the
    GPU's current E and Q as inputs; over the steps nothing is lost
    (sum of outputs + final memory = sum of gradients + initial memory)."""
    m, n, r = 600, 450, 10
    c0 = _case(m, n, r, 40, dtype)
    items = _items(pk, [c0], r, dtype)
    it = items[0]
    E0 = it["E"].double().cpu()
    sum_out = torch.zeros(m, n, dtype=torch.float64)
    sum_g = torch.zeros(m, n, dtype=torch.float64)
    for t in range(4):
        G = _case(m, n, r, 50 + t, dtype)["G"]
        c = dict(G=G, E=it["E"].cpu(), Q=it["Q"].cpu())
        it["G"] = G.cuda()
        pk.psgd_step(items, r, dtype)
        torch.cuda.synchronize()
        _check_step(c, _host(it), dtype, f"step {t}")
        sum_out += it["out"].double().cpu()
        sum_g += G.double()
    lhs = sum_out + it["E"].double().cpu()
    rhs = sum_g + E0
    # each step's E' = M - out is exact up to one fp32 rounding of M and of E'
    assert (lhs - rhs).abs().max().item() <= 16 * 2 ** -24 * rhs.abs().max().item()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_low_rank_gradient_is_reconstructed(pk, dtype):
    m, n, r = 333, 260, 8
    c = _case(m, n, r, 70, dtype, e_scale=0.0, rank=3)
    items = _items(pk, [c], r, dtype)
    pk.psgd_step(items, r, dtype)
    torch.cuda.synchronize()
    got = _host(items[0])
    G = c["G"].double()
    # rank 3 < r: the output is G up to the product's rounding; the rest of
    # P_hat is valid (orthonormal, orthogonal to the kept span) but not unique
    assert osp.rel_fro(got["out"].double().numpy(), G.numpy()) <= (2e-2 if dtype == torch.bfloat16 else 1e-5)
    P = got["P"].double()
    nz = P.norm(dim=0) > 0.5
    assert torch.allclose(P[:, nz].T @ P[:, nz], torch.eye(int(nz.sum()), dtype=torch.float64), atol=1e-3)
    M = (c["E"] + c["G"].float())
    assert torch.equal(got["E"], M - got["out"].float())


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_zero_gradient_and_memory(pk, dtype):
    m, n, r = 200, 136, 5
    c = dict(G=torch.zeros(m, n, dtype=dtype), E=torch.zeros(m, n), Q=workloads.gaussian((n, r), 1))
    items = _items(pk, [c], r, dtype)
    pk.psgd_step(items, r, dtype)
    torch.cuda.synchronize()
    for k in ("E", "P", "Q", "out"):
        assert torch.all(items[0][k] == 0), k


def test_many_matrices_fused_first_pass_and_in_place_output(pk):
    """Eighteen matrices in one call (two launches per kernel); 8192-row
    matrices whose row blocks fill the GPU take the fused first pass.  The
    output may overwrite G."""
    dtype = torch.bfloat16
    r = 16
    shapes = [(8192, 1024)] * 8 + [(64 + 24 * i, 200 + 8 * i) for i in range(10)]
    cases = [_case(m, n, r, 100 + i, dtype) for i, (m, n) in enumerate(shapes)]
    items = _items(pk, cases, r, dtype, out_is_g=True)
    pk.psgd_step(items, r, dtype)
    torch.cuda.synchronize()
    for i, (c, it) in enumerate(zip(cases, items)):
        _check_step(c, _host(it), dtype, f"matrix {i}")


def test_70b_class_mlp_matrix_full_size(pk):
    """One 8192 x 28672 MLP gradient of the 70B-class layer at the x64 rank
    (r = 99), bf16: P_hat and Q against the float64 oracle in full, the
    output and the memory on sampled rows."""
    cfg = workloads.CONFIGS[5]
    m, n = cfg.grad.shapes[1]
    r = ops.rank_for_ratio(m, n)
    dev = torch.device("cuda")
    _, G = workloads.grad_pair_fast(cfg.grad, 5, 0, 1, dev)
    gen = torch.Generator(device=dev).manual_seed(9)
    E = 0.05 * G.float().std() * torch.randn(m, n, device=dev, generator=gen)
    Q = torch.randn(n, r, device=dev, generator=gen)
    Gh, Eh, Qh = G.double().cpu().numpy(), E.double().cpu().numpy(), Q.double().cpu().numpy()
    items = [dict(G=G, E=E, P=torch.zeros(m, r, device=dev), Q=Q.clone(),
                  out=torch.empty(m, n, dtype=torch.bfloat16, device=dev), ws=pk.psgd_workspace(m, n, r, G.dtype, dev))]
    pk.psgd_step(items, r, torch.bfloat16)
    torch.cuda.synchronize()
    M = Gh + Eh
    P_hat = ops.gram_schmidt(M @ Qh)
    Qn = M.T @ P_hat
    got = items[0]
    assert osp.rel_fro(got["P"].double().cpu().numpy(), P_hat) <= 2e-2
    assert osp.rel_fro(got["Q"].double().cpu().numpy(), Qn) <= 2e-2
    rows = np.r_[0:16, m // 2:m // 2 + 16, m - 16:m]
    out_o = P_hat[rows] @ Qn.T
    out = got["out"][rows].double().cpu().numpy()
    assert osp.rel_fro(out, out_o) <= 2e-2
    Mr = (torch.from_numpy(Eh[rows]).float() + torch.from_numpy(Gh[rows]).float())
    assert torch.equal(got["E"][rows].cpu(), Mr - got["out"][rows].float().cpu())


def test_bad_arguments_leave_state_untouched(pk):
    dtype = torch.bfloat16
    c = _case(128, 96, 4, 3, dtype)
    items = _items(pk, [c], 4, dtype)
    before = {k: v.clone() for k, v in items[0].items()}
    with pytest.raises(pk.AcscError) as e:
        pk.psgd_step(items, 97, dtype)             # r > min(m, n)
    assert e.value.code == pk.ACSC_EINVAL
    small = dict(items[0], ws=items[0]["ws"][:1024])
    with pytest.raises(pk.AcscError) as e:
        pk.psgd_step([small], 4, dtype)
    assert e.value.code == pk.ACSC_ENOSPC
    torch.cuda.synchronize()
    for k in ("G", "E", "P", "Q"):
        assert torch.equal(items[0][k], before[k]), k
