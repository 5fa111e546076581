"""sc_correct_static (the correction on the library's own device scratch, for
callers that cannot allocate) against sc_correct with a caller workspace,
called through the C ABI: bit-identical outputs on two calls in a row, the
second on a smaller matrix (the scratch keeps the first call's contents), in
both dtypes, and a shape beyond the scratch refused before any launch."""
import ctypes as C

import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_14339_amd as pk
    return pk


def _prior(m, n, r, seed):
    U, s, V = workloads.random_orthonormal_basis(m, n, r, seed, "cuda")
    d = (s / (s + 0.7)).float()
    return U.float().contiguous(), d.contiguous(), V.float().contiguous()


def _static_call(pk, G, U, d, V, out, alpha):
    m, n = G.shape
    return pk.lib.sc_correct_static(pk._ptr(G), pk._dt(G), m, n, pk._ptr(U), pk._ptr(d), pk._ptr(V), U.shape[1],
                                    float(alpha), pk._ptr(out), pk._stream())


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_static_scratch_matches_the_workspace_call_on_two_calls(pk, dtype):
    alpha = workloads.ALPHA
    # first the largest 70B-class shape (88 MiB of the 96 MiB scratch), then
    # a smaller one: the second call finds the first call's bytes there
    shapes = [((28672, 8192, 128) if dtype == torch.bfloat16 else (8192, 8192, 128)), (1000, 2056, 40)]
    for i, (m, n, r) in enumerate(shapes):
        G = workloads.gaussian((m, n), seed=10 + i, device="cuda", dtype=dtype)
        U, d, V = _prior(m, n, r, 20 + i)
        ref = pk.sc_correct(G, U, d, V, alpha)
        out = torch.full_like(G, float("nan"))
        assert _static_call(pk, G, U, d, V, out, alpha) == 0, pk.lib.acsc_last_error()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), (m, n, r)
    # in place (G_proj == G), as sc_correct allows
    G2 = G.clone()
    assert _static_call(pk, G2, U, d, V, G2, alpha) == 0
    torch.cuda.synchronize()
    assert torch.equal(G2, ref)


def test_static_scratch_refuses_a_shape_beyond_its_size(pk):
    size = C.c_size_t(0)
    assert pk.lib.sc_adamw_workspace_size(65536, 8192, 128, pk.BF16, C.byref(size)) == 0
    assert size.value > pk.SC_STATIC_SCRATCH_BYTES
    G = torch.empty(0, dtype=torch.bfloat16, device="cuda")
    f = torch.empty(0, device="cuda")
    rc = pk.lib.sc_correct_static(pk._ptr(G), pk.BF16, 65536, 8192, pk._ptr(f), pk._ptr(f), pk._ptr(f), 128, 0.3,
                                  pk._ptr(G), pk._stream())
    assert rc == pk.ACSC_ENOSPC
    assert "scratch" in pk.lib.acsc_last_error().decode()
