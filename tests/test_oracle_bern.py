"""Pins of the Bernoulli mask oracle (paper App. F: each entry of the mask is
an independent Bernoulli draw; the receiver rescales by 1 / (1 - p)).

The per-entry draw is our specification, so nothing the paper prints pins
its values; it is pinned by what a Bernoulli mask must satisfy: inclusion
frequency per position, the binomial law of the row counts, independence of
neighbouring entries (including the two that share one hash), the uniform
law of all patterns on a tiny row, keep = 1, and the App. F propositions
(the rescaled mask is unbiased and its variance is (p / (1 - p)) h^2), plus
the layout invariants of the payload.
"""
import numpy as np
import pytest

from oracle import mask as om


def _key(i=0, H=256, S=64):
    return om.mask_key(7 + i, 2, 9, 1, 4, S, H)


def test_inclusion_frequency_and_row_counts():
    H, rows, keep = 256, 4096, 0.1
    q = om.bern_threshold(keep) / 65536
    m = om.bern_mask_dense(_key(), rows, H, keep)
    # per position: binomial(rows, q) frequencies, chi-square on H - 1 dof
    f = m.sum(axis=0)
    chi2 = np.sum((f - rows * q) ** 2 / (rows * q * (1 - q)))
    assert chi2 < H + 5 * np.sqrt(2 * H)
    # per row: binomial(H, q) counts
    c = m.sum(axis=1)
    assert abs(c.mean() - H * q) < 5 * np.sqrt(H * q * (1 - q) / rows)
    assert abs(c.var() / (H * q * (1 - q)) - 1) < 5 * np.sqrt(2 / rows)


@pytest.mark.parametrize("offset", [0, 1])
def test_neighbouring_entries_are_independent(offset):
    # offset 0: entries 2q, 2q + 1 (one hash, two halves); 1: 2q + 1, 2q + 2
    H, rows, keep = 256, 4096, 0.3
    q = om.bern_threshold(keep) / 65536
    m = om.bern_mask_dense(_key(1), rows, H, keep).astype(np.float64)
    a = m[:, offset:H - 1:2]
    b = m[:, offset + 1::2][:, :a.shape[1]]
    n = a.size
    both = np.mean(a * b)
    assert abs(both - q * q) < 5 * np.sqrt(q * q * (1 - q * q) / n)


def test_all_patterns_of_a_tiny_row_are_equally_likely():
    # H = 4, keep = 1/2: the 16 patterns with probability 1/16 each
    rows = 1 << 14
    m = om.bern_mask_dense(_key(2, H=4, S=rows), rows, 4, 0.5)
    code = m @ np.array([1, 2, 4, 8])
    f = np.bincount(code, minlength=16)
    chi2 = np.sum((f - rows / 16) ** 2 / (rows / 16))
    assert chi2 < 15 + 5 * np.sqrt(30)


def test_keep_one_keeps_everything_and_thresholds():
    assert om.bern_threshold(1.0) == 65536 and om.bern_threshold(0.02) == 1311
    m = om.bern_mask_dense(_key(3), 8, 100, 1.0)
    assert m.all()
    with pytest.raises(ValueError):
        om.bern_threshold(0.0)


def test_unbiased_and_variance_after_rescale():
    """App. F: E[h~] = h with h~ = h ⊙ m / (1 - p), and
    Var[h~_i] = (p / (1 - p)) h_i^2, over independent masks (keys)."""
    H, keep, trials = 64, 0.25, 4000
    q = om.bern_threshold(keep) / 65536
    h = np.linspace(-2.0, 3.0, H).astype(np.float32)
    acc = np.zeros(H)
    acc2 = np.zeros(H)
    for t in range(trials):
        k = om.mask_key(1000 + t, 0, 0, 0, 1, 1, H)
        rp, v, i = om.bern_pack(h[None, :], keep, k)
        y = om.bern_unpack(v, rp, H, k, keep, scale=1.0 / q).astype(np.float64)[0]
        acc += y
        acc2 += y * y
    mean = acc / trials
    var = acc2 / trials - mean ** 2
    p = 1.0 - q
    expect_var = (p / (1 - p)) * h.astype(np.float64) ** 2
    se = np.sqrt(expect_var / trials) + 1e-12
    assert np.all(np.abs(mean - h) <= 5 * se)
    nz = np.abs(h) > 0.3
    assert np.all(np.abs(var[nz] / expect_var[nz] - 1) < 0.2)


@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
def test_payload_layout_and_round_trip(dtype):
    rows, H, keep = 37, 300, 0.07
    rng = np.random.default_rng(5)
    x = rng.standard_normal((rows, H)).astype(np.float32)
    if dtype == np.uint16:
        x = (x.view(np.uint32) >> 16).astype(np.uint16)
    k = _key(4, H, rows)
    rp, v, i = om.bern_pack(x, keep, k)
    m = om.bern_mask_dense(k, rows, H, keep)
    assert rp[0] == 0 and np.all(np.diff(rp) == m.sum(axis=1))
    for r in range(rows):
        seg = i[rp[r]:rp[r + 1]].astype(np.int64)
        assert np.all(np.diff(seg) > 0) and np.array_equal(seg, np.nonzero(m[r])[0])
        assert np.array_equal(v[rp[r]:rp[r + 1]], x[r, seg])
    y = om.bern_unpack(v, rp, H, k, keep, scale=1.0)
    assert np.array_equal(y.view(np.uint8), np.where(m.astype(bool), x, 0).astype(x.dtype).view(np.uint8))
    y2 = om.bern_unpack(v, rp, H, k, keep, scale=1.0, idx=i)
    assert np.array_equal(y2, y)
    # rows sampled from the middle of a tensor carry their own offsets
    rp5, v5, i5 = om.bern_pack(x[5:9], keep, k, row0=5)
    assert np.array_equal(v5, v[rp[5]:rp[9]]) and np.array_equal(rp5, rp[5:10] - rp[5])
