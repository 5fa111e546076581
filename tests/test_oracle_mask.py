"""Pins of the masking-compressor oracle (paper Sec. 3.1; App. F; App. H).

Each check is something other than the oracle itself: published hash test
vectors, brute-force enumeration, sampling statistics, the paper's closed
forms and worked arithmetic, and torch's own bf16 rounding.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import mask as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
GAMMA = 0x9E3779B97F4A7C15
M64 = 2 ** 64 - 1


def _read_pairs(name):
    out = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                out.append(line.split())
    return out


def test_mix64_matches_published_splitmix64_stream():
    state = 0
    for (v,) in _read_pairs("splitmix64_seed0.txt"):
        state = (state + GAMMA) & M64
        assert om.mix64(state) == int(v, 16)


def test_fmix32_matches_murmur3_empty_input_vectors():
    for seed, h in _read_pairs("murmur3_fmix32.txt"):
        assert om.fmix32(int(seed, 16)) == int(h, 16)


@pytest.mark.parametrize("w", [2, 4, 6, 8, 10, 12, 14])
def test_feistel_is_a_bijection_on_its_domain(w):
    for rk in (0, 1, 0xDEADBEEFCAFEBABE, om.row_key(12345, 7)):
        img = {om.feistel(x, w, rk) for x in range(1 << w)}
        assert img == set(range(1 << w))


def test_domain_bits_is_smallest_even_power_covering_H():
    for H in [1, 2, 3, 4, 5, 16, 17, 255, 256, 257, 2048, 4096, 8192, 65536]:
        w = om.domain_bits(H)
        assert w % 2 == 0 and w >= 2 and (1 << w) >= H
        assert w == 2 or (1 << (w - 2)) < H


@pytest.mark.parametrize("H", [1, 2, 3, 5, 7, 8, 100, 255, 256, 257, 1000, 2047, 2048, 2049])
def test_cycle_walked_feistel_is_a_permutation_of_range_H(H):
    for rk in (3, om.row_key(99, H)):
        img = [om.perm(i, H, rk) for i in range(H)]
        assert sorted(img) == list(range(H))


def test_keep_count_rounds_half_up_and_validates():
    assert om.keep_count(2048, 0.05) == 102      # round(102.4)
    assert om.keep_count(256, 0.1) == 26         # round(25.6)
    assert om.keep_count(4096, 0.02) == 82       # round(81.92)
    assert om.keep_count(4096, 0.05) == 205      # round(204.8)
    assert om.keep_count(4096, 0.1) == 410       # round(409.6)
    assert om.keep_count(8192, 0.02) == 164      # round(163.84)
    assert om.keep_count(10, 0.25) == 3          # 2.5 -> 3 (half up)
    assert om.keep_count(7, 1.0) == 7
    for bad in (0.0, -0.1, 1.5, float("nan")):
        with pytest.raises(ValueError):
            om.keep_count(64, bad)
    with pytest.raises(ValueError):
        om.keep_count(10, 0.01)                  # K = 0


def test_indices_are_K_distinct_ascending_and_in_range():
    key = om.mask_key(7, 3, 11, 0, 2, 64, 300)
    idx = om.indices(key, 64, 300, 37)
    assert idx.shape == (64, 37)
    assert np.all(np.diff(idx.astype(np.int64), axis=1) > 0)
    assert idx.min() >= 0 and idx.max() < 300
    # full keep is the identity subset
    full = om.indices(key, 4, 300, 300)
    assert np.array_equal(full, np.tile(np.arange(300), (4, 1)))


def test_mask_is_deterministic_and_keyed_on_layer_step_microbatch_seed_and_shape():
    base = dict(seed=1, layer=2, step=3, microbatch=4, B=2, S=8, H=512)
    k0 = om.mask_key(**base)
    ref = om.indices(k0, 16, 512, 25)
    assert np.array_equal(ref, om.indices(om.mask_key(**base), 16, 512, 25))
    for field in ("seed", "layer", "step", "microbatch", "B", "S"):
        alt = dict(base)
        alt[field] += 1
        other = om.indices(om.mask_key(**alt), 16, 512, 25)
        assert not np.array_equal(ref, other), field
    # rows differ from each other
    assert len({tuple(r) for r in ref}) == 16


def test_two_of_eight_subsets_are_uniform():
    # brute force: every one of the C(8,2) = 28 subsets, over 1e5 row keys
    H, K, n = 8, 2, 100_000
    key = om.mask_key(2609, 0, 1, 0, 1, n, H)
    idx = om.indices(key, n, H, K)
    code = idx[:, 0] * 8 + idx[:, 1]
    counts = np.bincount(code, minlength=64)
    pairs = [a * 8 + b for a in range(8) for b in range(a + 1, 8)]
    obs = counts[pairs]
    assert obs.sum() == n
    exp = n / 28.0
    chi2 = float(((obs - exp) ** 2 / exp).sum())
    # 27 degrees of freedom: P(chi2 > 70) ~ 1e-5
    assert chi2 < 70.0, (chi2, obs)


def test_inclusion_and_pairwise_frequencies_match_uniform_K_subsets():
    H, K, rows = 2048, 102, 16384
    key = om.mask_key(14341, 0, 1, 0, 8, 2048, H)
    m = om.mask_dense(key, rows, H, K).astype(np.float64)
    assert np.all(m.sum(axis=1) == K)
    p = K / H
    col = m.sum(axis=0)
    chi2 = float(((col - rows * p) ** 2 / (rows * p * (1 - p))).sum())
    # 2047 dof: mean 2047, sd 64; reject beyond 6 sd
    assert abs(chi2 - (H - 1)) < 6 * math.sqrt(2 * (H - 1)), chi2
    # pairwise inclusion K(K-1)/(H(H-1)) for a few fixed and adjacent pairs
    q = K * (K - 1) / (H * (H - 1))
    for a, b in [(0, 1), (5, 6), (100, 2047), (1023, 1024), (7, 1500)]:
        both = float((m[:, a] * m[:, b]).sum())
        sd = math.sqrt(rows * q * (1 - q))
        assert abs(both - rows * q) < 5 * sd + 1, (a, b, both, rows * q)


def _rand_bf16_bits(shape, seed):
    t = torch.randn(*shape, generator=torch.Generator().manual_seed(seed)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pack_unpack_round_trip_is_x_times_mask(dtype):
    rows, H, K = 40, 333, 50
    key = om.mask_key(5, 1, 2, 3, 4, 10, H)
    if dtype == "f32":
        x = np.random.default_rng(0).standard_normal((rows, H)).astype(np.float32)
    else:
        x = _rand_bf16_bits((rows, H), 0)
    vals, idx = om.pack(x, K, key)
    m = om.mask_dense(key, rows, H, K).astype(bool)
    # packed values are the kept entries in ascending column order (bit copies)
    for r in range(rows):
        assert np.array_equal(idx[r], np.nonzero(m[r])[0])
        assert np.array_equal(vals[r].view(np.uint8), x[r, m[r]].view(np.uint8))
    y = om.unpack(vals, H, key, 1.0)
    expect = np.where(m, x, np.zeros_like(x))
    assert np.array_equal(y.view(np.uint8), expect.view(np.uint8))
    # off-mask entries are +0 (all-zero bit patterns)
    assert np.all(y.view(np.uint8).reshape(rows, H, -1)[~m] == 0)
    # idx-driven unpack equals key-driven unpack
    y2 = om.unpack(vals, H, key, 1.0, idx=idx)
    assert np.array_equal(y.view(np.uint8), y2.view(np.uint8))
    # pack . unpack . pack == pack (idempotent on the payload)
    v2, i2 = om.pack(y, K, key)
    assert np.array_equal(v2.view(np.uint8), vals.view(np.uint8)) and np.array_equal(i2, idx)


def test_pack_rows_are_global_token_indices():
    rows, H, K = 12, 64, 9
    key = om.mask_key(1, 0, 0, 0, 3, 4, H)
    x = np.random.default_rng(1).standard_normal((rows, H)).astype(np.float32)
    full, _ = om.pack(x, K, key)
    tail, _ = om.pack(x[5:], K, key, row0=5)
    assert np.array_equal(full[5:], tail)


def test_unpack_scale_fp32_is_one_ieee_multiply():
    rows, H, K = 16, 128, 31
    key = om.mask_key(9, 0, 0, 0, 1, 16, H)
    x = np.random.default_rng(2).standard_normal((rows, H)).astype(np.float32) * 37.0
    vals, _ = om.pack(x, K, key)
    scale = np.float32(H / K)
    y = om.unpack(vals, H, key, float(scale))
    m = om.mask_dense(key, rows, H, K).astype(bool)
    assert np.array_equal(y[m], (vals.reshape(-1) * scale).astype(np.float32))


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    g = torch.Generator().manual_seed(3)
    f = torch.randn(200_000, generator=g) * torch.exp(torch.randn(200_000, generator=g) * 8)
    # add exact ties and near-ties of the bf16 grid
    base = torch.randn(2000, generator=g).to(torch.bfloat16).float()
    ulp_half = base.abs() * 2.0 ** -8
    f = torch.cat([f, base + ulp_half, base - ulp_half, torch.tensor([1 + 2 ** -8, 1 + 3 * 2 ** -8,
                                                                       -1 - 2 ** -8, 3e38, 1e-40,
                                                                       -1e-41, 0.0, -0.0])])
    f = f.to(torch.float32)
    ref = f.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([om.bf16_from_double(float(v)) for v in f.tolist()], dtype=np.uint16)
    assert np.array_equal(got, ref)
    assert om.bf16_from_double(1 + 2 ** -8) == 0x3F80       # tie -> even
    assert om.bf16_from_double(1 + 3 * 2 ** -8) == 0x3F82   # tie -> even (up)
    for h in (0x3F80, 0xC0A0, 0x0001, 0x7F7F):
        assert om.bf16_from_double(om.bf16_to_double(h)) == h


def test_bf16_scale_is_rounded_once_from_the_exact_product():
    # exact product of a bf16 value and an fp32 scale lies between two bf16
    # numbers; rounding it once can differ from rounding through fp32 first
    v = 1.0 + 2 ** -7                 # bf16 value 0x3F81
    s = 1.0 - 2 ** -24 * 3            # fp32 scale just below 1
    p = v * s                         # exact in double
    via_f32 = float(np.float32(p))
    once = om.bf16_from_double(p)
    assert once == 0x3F81             # the exact product is below 1 + 2^-7 by a hair
    assert om.bf16_from_double(via_f32) in (0x3F81, 0x3F80)


def test_rescaled_mask_is_unbiased_with_fixed_K_variance():
    # App. F: E[h_tilde] = h after rescaling; per-coordinate variance.  With a
    # fixed K per token and scale H/K, E = h and Var = (H/K - 1) h^2.
    H, K, rows = 64, 16, 40_000
    h = np.linspace(-2.0, 3.0, H).astype(np.float32)
    x = np.tile(h, (rows, 1))
    key = om.mask_key(11, 0, 0, 0, 1, rows, H)
    vals, _ = om.pack(x, K, key, with_idx=False)
    y = om.unpack(vals, H, key, float(np.float32(H / K))).astype(np.float64)
    mean = y.mean(axis=0)
    var = y.var(axis=0)
    theo_var = (H / K - 1.0) * h.astype(np.float64) ** 2
    se = np.sqrt(theo_var / rows) + 1e-12
    assert np.all(np.abs(mean - h) <= 5 * se + 1e-6)
    nz = np.abs(h) > 0.2
    assert np.all(np.abs(var[nz] / theo_var[nz] - 1.0) < 0.06)


def test_paper_worked_payload_arithmetic():
    g = dict((k, float(v)) for k, v in _read_pairs("paper_pp_payload.txt"))
    S, H, b = int(g["S"]), int(g["H"]), int(g["bytes_per_elem"])
    dense = S * H * b
    assert dense == int(g["boundary_MB"]) * 2 ** 20            # "8 MB"
    step = g["boundaries"] * g["microbatches"] * g["directions"] * dense
    assert abs(step / 1e9 - g["step_GB"]) < 0.1                 # "about 1.8 GB"
    K = om.keep_count(H, round(1.0 - g["p"], 12))
    key = om.mask_key(0, 0, 1, 0, 1, S, H)
    x = np.zeros((4, H), dtype=np.uint16)
    vals, _ = om.pack(x, K, key, with_idx=False)
    frac = vals.nbytes / x.nbytes
    assert abs(frac - g["masked_fraction"]) < 0.001              # "5% of the volume"


def test_paper_defaults_fixture_agrees_with_workloads():
    import workloads
    g = dict((k, float(v)) for k, v in _read_pairs("paper_defaults.txt"))
    assert workloads.ALPHA == g["alpha"] and workloads.TAU == g["tau"]
    assert workloads.CONFIGS[2].act.keep == (round(1 - g["p"], 12),)


@pytest.mark.parametrize("H,K,rows", [(256, 26, 40_000), (2048, 102, 16_384), (8192, 164, 8_192)])
def test_structured_pair_classes_show_no_correlation(H, K, rows):
    # Feistel structure could correlate positions that share a half (offset
    # 2^(w/2)), neighbours (offset 1) or distant halves (offset H/2).
    key = om.mask_key(77, 1, 2, 0, 1, rows, H)
    m = om.mask_dense(key, rows, H, K)
    q = K * (K - 1) / (H * (H - 1))
    w = om.domain_bits(H)
    for d in (1, 2, 1 << (w // 2), H // 2):
        cnt = int((m[:, :-d] & m[:, d:]).sum(dtype=np.int64))
        exp = q * rows * (H - d)
        # co-occurrence counts over distinct pairs are nearly independent
        z = (cnt - exp) / math.sqrt(exp)
        assert abs(z) < 5.0, (d, z)
