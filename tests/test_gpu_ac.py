"""GPU parity of the masking compressor against the CPU oracle (Sec. 3.1; App. F).

Indices and packed layouts are compared bit for bit; unpacked outputs too,
since the scaled value is defined as the exact product rounded once (bf16
results in the fp32 normal range).  Sizes cover the five workloads at full
size (the oracle is plain C and fast enough), plus ragged and edge shapes.
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
    return t.view(torch.int32).numpy().view(np.uint32)


def _host_x(x: torch.Tensor) -> np.ndarray:
    return _bits(x) if x.dtype == torch.bfloat16 else x.cpu().numpy()


def _run_case(pk, x_cpu: torch.Tensor, B, S, H, K, key_fields, scales=(1.0,), check_rows=None,
              ld_pad=0):
    """Pack / unpack on the GPU and compare with the oracle, bit for bit."""
    rows = B * S
    dev = torch.device("cuda")
    if ld_pad:
        big = torch.zeros(rows, H + ld_pad, dtype=x_cpu.dtype)
        big[:, :H] = x_cpu
        xg = big.to(dev)[:, :H]
    else:
        xg = x_cpu.to(dev)
    key = pk.make_key(B=B, S=S, H=H, **key_fields)
    okey = om.mask_key(key_fields["seed"], key_fields["layer"], key_fields["step"],
                       key_fields["microbatch"], B, S, H)
    vals, idx = pk.ac_mask_pack(xg, K, key)
    vals2, none = pk.ac_mask_pack(xg, K, key, with_idx=False)
    assert none is None
    torch.cuda.synchronize()
    xh = _host_x(x_cpu)
    sel = np.arange(rows) if check_rows is None else np.asarray(check_rows)
    if check_rows is None:
        ov, oi = om.pack(xh, K, okey)
    else:
        ov = np.concatenate([om.pack(xh[r:r + 1], K, okey, row0=int(r))[0] for r in sel])
        oi = np.concatenate([om.pack(xh[r:r + 1], K, okey, row0=int(r))[1] for r in sel])
    gv, gi = _bits(vals)[sel], _bits(idx)[sel]
    assert np.array_equal(gi, oi), "indices differ"
    assert np.array_equal(gv.view(np.uint8), ov.view(np.uint8)), "packed values differ"
    assert np.array_equal(_bits(vals2), _bits(vals)), "values-only pack differs"
    for scale in scales:
        y = pk.ac_unpack_scatter(vals, H, key, scale=scale)
        y2 = pk.ac_unpack_scatter(vals, H, key, scale=scale, idx=idx)
        torch.cuda.synchronize()
        vh = _bits(vals)
        if vals.dtype == torch.float32:
            vh = vh.view(np.float32)
        if check_rows is None:
            oy = om.unpack(vh, H, okey, scale)
        else:
            oy = np.concatenate([om.unpack(vh[r:r + 1], H, okey, scale, row0=int(r)) for r in sel])
        gy = _bits(y)[sel]
        assert np.array_equal(gy.view(np.uint8), oy.view(np.uint8)), f"unpack differs, scale={scale}"
        assert np.array_equal(_bits(y2), _bits(y)), f"idx-driven unpack differs, scale={scale}"
    return vals, idx


def _cfg_act(cid, rows=None, tensor_id=0):
    spec = workloads.CONFIGS[cid].act
    return workloads.activation(spec, cid, 0, tensor_id, "cpu", rows=rows)


@pytest.mark.parametrize("cid", [1, 2])
def test_config_full_size_bit_exact(pk, cid):
    spec = workloads.CONFIGS[cid].act
    x = _cfg_act(cid)
    for keep in spec.keep:
        K = om.keep_count(spec.H, keep)
        _run_case(pk, x, spec.B, spec.S, spec.H, K, workloads.mask_key_fields(cid),
                  scales=(1.0, spec.H / K))


@pytest.mark.parametrize("keep", [0.02, 0.05, 0.1])
def test_8b_heavy_tailed_full_size_bit_exact(pk, keep):
    spec = workloads.CONFIGS[3].act
    x = _cfg_act(3)
    K = om.keep_count(spec.H, keep)
    _run_case(pk, x, spec.B, spec.S, spec.H, K, workloads.mask_key_fields(3),
              scales=(spec.H / K,))


@pytest.mark.parametrize("layer", [0, 3])
def test_70b_slice_forward_and_backward_share_the_mask(pk, layer):
    spec = workloads.CONFIGS[5].act
    K = om.keep_count(spec.H, spec.keep[0])
    fields = workloads.mask_key_fields(5, layer=layer)
    x = _cfg_act(5, tensor_id=2 * layer)          # activation
    gx = _cfg_act(5, tensor_id=2 * layer + 1)     # activation gradient
    rows = spec.B * spec.S
    check = np.r_[0:64, rows // 2 - 3:rows // 2 + 61, rows - 64:rows]
    _, idx_f = _run_case(pk, x, spec.B, spec.S, spec.H, K, fields, scales=(spec.H / K,),
                         check_rows=check)
    _, idx_b = _run_case(pk, gx, spec.B, spec.S, spec.H, K, fields, scales=(spec.H / K,),
                         check_rows=check)
    assert torch.equal(idx_f, idx_b)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,S,H,K", [(1, 1, 1, 1), (3, 7, 13, 5), (2, 33, 333, 50),
                                     (1, 9, 1000, 1000), (2, 5, 2049, 1), (1, 65, 4097, 410),
                                     (1, 3, 65536, 1311), (1, 2, 16, 16), (5, 13, 17, 3)])
def test_ragged_and_edge_shapes(pk, dtype, B, S, H, K):
    x = workloads.gaussian((B * S, H), seed=H * 31 + K, dtype=dtype)
    fields = dict(seed=99, layer=1, step=7, microbatch=2)
    _run_case(pk, x, B, S, H, K, fields, scales=(1.0, H / K, -0.75))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_strided_rows_and_unaligned_output(pk, dtype):
    B, S, H, K = 2, 40, 300, 33
    x = workloads.gaussian((B * S, H), seed=5, dtype=dtype)
    fields = dict(seed=3, layer=0, step=1, microbatch=0)
    _run_case(pk, x, B, S, H, K, fields, ld_pad=13)
    # output with an odd row stride takes the element-wise store path
    key = pk.make_key(B=B, S=S, H=H, **fields)
    vals, idx = pk.ac_mask_pack(x.cuda(), K, key)
    ybig = torch.full((B * S, H + 3), 7.0, dtype=dtype, device="cuda")
    y = pk.ac_unpack_scatter(vals, H, key, scale=2.0, y=ybig[:, :H])
    ref = pk.ac_unpack_scatter(vals, H, key, scale=2.0)
    torch.cuda.synchronize()
    assert torch.equal(y, ref)
    assert torch.all(ybig[:, H:] == 7.0)     # columns past H untouched


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("H,K,pad", [(301, 100, 3), (2045, 400, 3), (9000, 3000, 8)])
def test_padded_rows_with_ragged_tail(pk, dtype, H, K, pad):
    # 16-byte aligned row stride with H not a multiple of the 16-byte chunk:
    # the whole-row pack reads the chunks, then the last few entries one by one
    B, S = 2, 9
    x = workloads.gaussian((B * S, H), seed=H + K, dtype=dtype)
    _run_case(pk, x, B, S, H, K, dict(seed=11, layer=2, step=5, microbatch=1), ld_pad=pad,
              scales=(1.0, H / K))


def test_zero_rows_and_determinism(pk):
    key0 = pk.make_key(seed=1, layer=0, step=0, microbatch=0, B=0, S=4, H=64)
    x = torch.empty(0, 64, device="cuda")
    v, i = pk.ac_mask_pack(x, 8, key0)
    assert v.shape == (0, 8)
    y = pk.ac_unpack_scatter(v, 64, key0)
    assert y.shape == (0, 64)
    spec = workloads.CONFIGS[2].act
    x = _cfg_act(2, rows=2048).cuda()
    key = pk.make_key(B=1, S=2048, H=spec.H, **workloads.mask_key_fields(2))
    a = pk.ac_mask_pack(x, 102, key)
    b = pk.ac_mask_pack(x, 102, key)
    ya = pk.ac_unpack_scatter(a[0], spec.H, key, 20.0)
    yb = pk.ac_unpack_scatter(b[0], spec.H, key, 20.0)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1]) and torch.equal(ya, yb)


def test_errors_raise_without_side_effects(pk):
    key = pk.make_key(seed=1, layer=0, step=0, microbatch=0, B=2, S=4, H=64)
    x = torch.randn(8, 64, device="cuda")
    vals = torch.full((8, 4), 3.0, device="cuda")
    with pytest.raises(pk.AcscError) as e:
        pk.ac_mask_pack(x, 65, key, vals=vals)
    assert e.value.code == pk.ACSC_EINVAL
    torch.cuda.synchronize()
    assert torch.all(vals == 3.0)


def _oracle_key(fields, B, S, H, layer):
    return om.mask_key(fields["seed"], layer, fields["step"], fields["microbatch"], B, S, H)


def test_70b_slice_all_rows_batched_index_list_flow(pk):
    """C5, every row of all four boundaries, both directions, in the batched
    launch configuration the benchmark times: the sender packs the activation
    from the key and keeps the index lists; the receiver unpacks from the key
    (values-only wire) and keeps its own lists; the receiver packs the
    activation gradient from its lists; the sender unpacks that payload from
    its lists.  Every array bit-exact against the oracle, both sides' lists
    equal, and boundary 2 equal to the single calls."""
    spec = workloads.CONFIGS[5].act
    H, rows, nl = spec.H, spec.B * spec.S, 4
    K = om.keep_count(H, spec.keep[0])
    fields = workloads.mask_key_fields(5, layer=0)
    key = pk.make_key(B=spec.B, S=spec.S, H=H, **fields)
    x = torch.stack([workloads.activation(spec, 5, 0, 2 * l, "cuda") for l in range(nl)])
    gx = torch.stack([workloads.activation(spec, 5, 0, 2 * l + 1, "cuda") for l in range(nl)])
    scale = H / K
    idx_s = torch.empty(nl, rows, K, dtype=torch.int16, device="cuda")
    idx_r = torch.empty_like(idx_s)
    vals = pk.ac_mask_pack_batched(x, K, key, idx_out=idx_s)
    y = pk.ac_unpack_scatter_batched(vals, H, key, scale, idx_out=idx_r)
    gvals = pk.ac_mask_pack_batched(gx, K, key, idx_in=idx_r)
    gy = pk.ac_unpack_scatter_batched(gvals, H, key, scale, idx_in=idx_s)
    torch.cuda.synchronize()
    assert torch.equal(idx_s, idx_r)
    for l in range(nl):
        okey = _oracle_key(fields, spec.B, spec.S, H, l)
        ov, oi = om.pack(_bits(x[l]), K, okey)
        assert np.array_equal(_bits(idx_s[l]), oi), l
        assert np.array_equal(_bits(vals[l]), ov), l
        assert np.array_equal(_bits(y[l]), om.unpack(ov, H, okey, scale)), l
        gov, goi = om.pack(_bits(gx[l]), K, okey)
        assert np.array_equal(goi, oi), l                         # backward inherits the mask
        assert np.array_equal(_bits(gvals[l]), gov), l
        assert np.array_equal(_bits(gy[l]), om.unpack(gov, H, okey, scale)), l
    k2 = pk.make_key(B=spec.B, S=spec.S, H=H, **workloads.mask_key_fields(5, layer=2))
    v2, i2 = pk.ac_mask_pack(x[2], K, k2)
    y2 = pk.ac_unpack_scatter(v2, H, k2, scale)
    torch.cuda.synchronize()
    assert torch.equal(v2, vals[2]) and torch.equal(i2, idx_s[2]) and torch.equal(y2, y[2])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("nl,B,S,H,K,pad", [(3, 2, 33, 333, 50, 0), (2, 1, 9, 1000, 1000, 8), (3, 5, 13, 17, 3, 3),
                                            (2, 1, 65, 4097, 410, 8), (1, 2, 3, 65536, 40000, 0),
                                            (2, 2, 40, 300, 300, 0), (4, 1, 1, 1, 1, 0)])
def test_batched_ragged_shapes_match_single_calls_and_oracle(pk, dtype, nl, B, S, H, K, pad):
    """Ragged rows, padded row strides, a dense keep (K = H, the whole-row
    pack), K > H / 4, and an unpack too large for its staged form (H = 65536,
    K = 40000): each boundary of a batched call bit-exact against the oracle
    and the single call, through both the key-driven and the index-driven
    forms, with layer strides wider than the tensors."""
    rows = B * S
    fields = dict(seed=77, layer=5, step=3, microbatch=1)
    key = pk.make_key(B=B, S=S, H=H, **fields)
    gap = 24                                    # spare rows between boundaries
    x_all = workloads.gaussian((nl * (rows + gap), H + pad), seed=H + K + nl, dtype=dtype).cuda()
    x = x_all.view(nl, rows + gap, H + pad)[:, :rows, :H]
    vals = torch.full((nl, rows + 1, K), 9, dtype=dtype, device="cuda")[:, :rows]
    idx_s = torch.empty(nl, rows + 2, K, dtype=torch.int16, device="cuda")[:, :rows]
    idx_r = torch.empty_like(idx_s)
    ybuf = torch.full((nl, rows + 3, H + pad), 7, dtype=dtype, device="cuda")
    y = ybuf[:, :rows, :H]
    pk.ac_mask_pack_batched(x, K, key, vals=vals, idx_out=idx_s)
    pk.ac_unpack_scatter_batched(vals, H, key, -0.75, idx_out=idx_r, y=y)
    vals_i = pk.ac_mask_pack_batched(x, K, key, idx_in=idx_r)
    y_i = pk.ac_unpack_scatter_batched(vals_i, H, key, -0.75, idx_in=idx_s)
    torch.cuda.synchronize()
    assert torch.all(ybuf[:, rows:] == 7) and (pad == 0 or torch.all(ybuf[:, :, H:] == 7))
    assert torch.equal(idx_s, idx_r) and torch.equal(vals_i, vals) and torch.equal(y_i, y)
    for l in range(nl):
        okey = _oracle_key(fields, B, S, H, l + 5)
        xl = x[l].cpu()
        ov, oi = om.pack(_host_x(xl), K, okey)
        assert np.array_equal(_bits(idx_s[l]), oi)
        assert np.array_equal(_bits(vals[l]).view(np.uint8), ov.view(np.uint8))
        vh = _bits(vals[l])
        if dtype == torch.float32:
            vh = vh.view(np.float32)
        oy = om.unpack(vh, H, okey, -0.75)
        assert np.array_equal(_bits(y[l]).view(np.uint8), oy.view(np.uint8))
        kl = pk.make_key(B=B, S=S, H=H, **dict(fields, layer=5 + l))
        v1, i1 = pk.ac_mask_pack(x[l], K, kl)
        y1 = pk.ac_unpack_scatter(v1, H, kl, -0.75)
        torch.cuda.synchronize()
        assert torch.equal(v1, vals[l]) and torch.equal(i1, idx_s[l]) and torch.equal(y1, y[l])


def test_index_driven_pack_reads_nothing_past_H(pk):
    """An index entry >= H packs +0 (the row is never read there)."""
    B, S, H, K = 1, 4, 100, 5
    key = pk.make_key(seed=1, layer=0, step=1, microbatch=0, B=B, S=S, H=H)
    x = (torch.arange(B * S * H, dtype=torch.float32, device="cuda") + 1).view(1, B * S, H)
    idx = torch.tensor([[0, 7, 99, 100, 32767]] * (B * S), dtype=torch.int16, device="cuda").view(1, B * S, K)
    v = pk.ac_mask_pack_batched(x, K, key, idx_in=idx)
    torch.cuda.synchronize()
    row0 = torch.arange(B * S, device="cuda").view(-1, 1) * H
    expect = torch.stack([row0[:, 0] + 1, row0[:, 0] + 8, row0[:, 0] + 100,
                          torch.zeros_like(row0[:, 0]), torch.zeros_like(row0[:, 0])], 1).float()
    assert torch.equal(v[0], expect)
