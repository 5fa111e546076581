"""GPU parity of the Bernoulli mask variant (paper App. F) against the CPU
oracle, bit for bit: row offsets, bitmaps, packed values and indices, and
unpacked rows (one rounding of the scaled value, as the fixed-K unpack).
Sizes: the 1B-class activation whole, sampled rows of a 70B-class layer,
ragged and edge shapes; a short payload capacity never writes past its end.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import mask as om

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_14339_amd as pk
    return pk


def _bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.int16:
        return t.numpy().view(np.uint16)
    if t.dtype == torch.int32:
        return t.numpy().view(np.uint32)
    return t.view(torch.int32).numpy().view(np.uint32)


def _host(t):
    return _bits(t) if t.dtype == torch.bfloat16 else t.cpu().numpy()


def _dense_from_bits(words: np.ndarray, H: int) -> np.ndarray:
    rows = words.shape[0]
    b = np.unpackbits(words.astype('<u4').view(np.uint8).reshape(rows, -1), axis=1, bitorder="little")
    return b[:, :H]


def _check(pk, x, B, S, H, keep, fields, rows_check=None, scales=(1.0,), ld_pad=0):
    dev = torch.device("cuda")
    rows = B * S
    if ld_pad:
        big = torch.zeros(rows, H + ld_pad, dtype=x.dtype)
        big[:, :H] = x
        xg = big.to(dev)[:, :H]
    else:
        xg = x.to(dev)
    key = pk.make_key(B=B, S=S, H=H, **fields)
    okey = om.mask_key(fields["seed"], fields["layer"], fields["step"], fields["microbatch"], B, S, H)
    rp, bits = pk.ac_bern_mask(rows, H, keep, key)
    vals, idx = pk.ac_bern_pack(xg, rp, bits)
    torch.cuda.synchronize()
    rp_h = rp.cpu().numpy()
    xh = _host(x)
    sel = np.arange(rows) if rows_check is None else np.asarray(rows_check)
    if rows_check is None:
        orp, ov, oi = om.bern_pack(xh, keep, okey)
        assert np.array_equal(rp_h, orp), "row offsets differ"
        m = om.bern_mask_dense(okey, rows, H, keep) if rows * H <= 1 << 16 else None
        if m is not None:
            assert np.array_equal(_dense_from_bits(_bits(bits), H), m), "bitmaps differ"
        assert np.array_equal(_bits(vals).view(np.uint8), ov.view(np.uint8)), "packed values differ"
        assert np.array_equal(_bits(idx), oi), "indices differ"
    else:
        for r in sel:
            r = int(r)
            orp, ov, oi = om.bern_pack(xh[r:r + 1], keep, okey, row0=r)
            a, b = rp_h[r], rp_h[r + 1]
            assert b - a == orp[1], f"row {r}: count differs"
            assert np.array_equal(_bits(vals[a:b]).view(np.uint8), ov.view(np.uint8)), f"row {r}: values differ"
            assert np.array_equal(_bits(idx[a:b]), oi), f"row {r}: indices differ"
    for scale in scales:
        y = pk.ac_bern_unpack(vals, H, rp, bits, scale)
        torch.cuda.synchronize()
        vh = _host(vals)
        gy = _bits(y)
        for r in (sel if rows_check is not None else [None]):
            if r is None:
                oy = om.bern_unpack(vh, rp_h, H, okey, keep, scale)
                assert np.array_equal(gy.view(np.uint8), oy.view(np.uint8)), f"unpack differs, scale={scale}"
            else:
                r = int(r)
                a, b = rp_h[r], rp_h[r + 1]
                oy = om.bern_unpack(vh[a:b], np.array([0, b - a]), H, okey, keep, scale, row0=r)
                assert np.array_equal(gy[r:r + 1].view(np.uint8), oy.view(np.uint8)), f"row {r}: unpack differs"
    return rp_h, vals


def test_1b_class_activation_whole(pk):
    spec = workloads.CONFIGS[2].act
    x = workloads.activation(spec, 2, 0, 0, "cpu")
    q = om.bern_threshold(0.05) / 65536
    _check(pk, x, spec.B, spec.S, spec.H, 0.05, workloads.mask_key_fields(2), scales=(1.0, 1.0 / q))


def test_70b_class_layer_sampled_rows(pk):
    spec = workloads.CONFIGS[5].act
    x = workloads.activation(spec, 5, 1, 0, "cpu")
    rows = spec.B * spec.S
    check = np.r_[0:32, rows // 2:rows // 2 + 32, rows - 32:rows]
    rp, vals = _check(pk, x, spec.B, spec.S, spec.H, 0.02, workloads.mask_key_fields(5, layer=1),
                      rows_check=check, scales=(50.0,))
    # the total count is binomial(rows * H, q)
    q = om.bern_threshold(0.02) / 65536
    n = rows * spec.H
    assert abs(rp[-1] - n * q) < 6 * np.sqrt(n * q * (1 - q))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,S,H,keep", [(1, 1, 1, 1.0), (3, 7, 13, 0.5), (2, 33, 31, 0.3), (1, 40, 33, 0.07),
                                        (2, 9, 300, 0.001), (1, 17, 2049, 0.2), (1, 3, 65536, 0.01),
                                        (2, 5, 64, 1.0)])
def test_ragged_and_edge_shapes(pk, dtype, B, S, H, keep):
    x = workloads.gaussian((B * S, H), seed=H * 7 + B, dtype=dtype)
    _check(pk, x, B, S, H, keep, dict(seed=11, layer=2, step=5, microbatch=1), scales=(1.0, -0.75, 3.0))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_strided_input_and_unaligned_output(pk, dtype):
    B, S, H, keep = 2, 24, 300, 0.1
    x = workloads.gaussian((B * S, H), seed=9, dtype=dtype)
    _check(pk, x, B, S, H, keep, dict(seed=3, layer=0, step=1, microbatch=0), ld_pad=13)
    key = pk.make_key(B=B, S=S, H=H, seed=3, layer=0, step=1, microbatch=0)
    rp, bits = pk.ac_bern_mask(B * S, H, keep, key)
    vals, _ = pk.ac_bern_pack(x.cuda(), rp, bits)
    ybig = torch.full((B * S, H + 3), 7.0, dtype=dtype, device="cuda")
    y = pk.ac_bern_unpack(vals, H, rp, bits, 2.0, y=ybig[:, :H])
    ref = pk.ac_bern_unpack(vals, H, rp, bits, 2.0)
    torch.cuda.synchronize()
    assert torch.equal(y, ref) and torch.all(ybig[:, H:] == 7.0)


def test_zero_rows_short_capacity_and_errors(pk):
    key0 = pk.make_key(seed=1, layer=0, step=0, microbatch=0, B=0, S=4, H=64)
    rp, bits = pk.ac_bern_mask(0, 64, 0.5, key0)
    torch.cuda.synchronize()
    assert rp.cpu().tolist() == [0]
    # a payload buffer shorter than nnz: nothing is written past its end
    B, S, H = 1, 64, 256
    key = pk.make_key(B=B, S=S, H=H, seed=2, layer=0, step=0, microbatch=0)
    x = workloads.gaussian((S, H), seed=2).cuda()
    rp, bits = pk.ac_bern_mask(S, H, 0.25, key)
    nnz = int(rp[-1].item())
    buf = torch.full((nnz,), -9.0, device="cuda")
    cap = nnz // 2
    rc = pk.lib.ac_bern_pack(pk._ptr(x), pk.F32, S, H, H, pk._ptr(rp), pk._ptr(bits), pk._ptr(buf), None, cap,
                             pk._stream())
    assert rc == 0
    full, _ = pk.ac_bern_pack(x, rp, bits)
    torch.cuda.synchronize()
    assert torch.equal(buf[:cap], full[:cap]) and torch.all(buf[cap:] == -9.0)
    # unpack with a short capacity reads zeros past it
    y = pk.ac_bern_unpack(full[:cap], H, rp, bits, 1.0)
    yf = pk.ac_bern_unpack(full, H, rp, bits, 1.0)
    torch.cuda.synchronize()
    m = yf != 0
    assert torch.all((y == yf) | (y == 0)) and int(y.ne(0).sum()) <= cap
    whole = int(np.searchsorted(rp.cpu().numpy()[1:], cap, side="right"))   # rows entirely below cap
    assert torch.equal(y[:whole], yf[:whole])
    with pytest.raises(pk.AcscError) as e:
        pk.ac_bern_mask(S, H, 0.0, key)
    assert e.value.code == pk.ACSC_EINVAL
    bad = pk.make_key(B=B, S=S, H=H + 1, seed=2, layer=0, step=0, microbatch=0)
    with pytest.raises(pk.AcscError):
        pk.ac_bern_mask(S, H, 0.5, bad)
    assert int(m.sum()) == nnz
