"""Seeded input generators: determinism and distribution checks (CPU)."""
import numpy as np
import pytest

import fixtures as F
from fixtures import workloads as WL

G = 0x9e3779b97f4a7c15


def _golden(golden_dir):
    vals = []
    with open(f"{golden_dir}/splitmix64_state0.txt") as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                vals.append(int(line, 16))
    return vals


def test_hash_matches_published_splitmix64(golden_dir):
    for k, ref in enumerate(_golden(golden_dir)):
        assert F.hash_u64(0, (k * G) % 2**64) == ref


def test_rmat_deterministic_simple():
    s1, d1 = F.rmat_edges(7, 4096, 20000, 0.57, 0.19, 0.19)
    s2, d2 = F.rmat_edges(7, 4096, 20000, 0.57, 0.19, 0.19)
    assert np.array_equal(s1, s2) and np.array_equal(d1, d2)
    s3, _ = F.rmat_edges(8, 4096, 20000, 0.57, 0.19, 0.19)
    assert not np.array_equal(s1, s3)
    assert (s1 != d1).all()
    key = s1.astype(np.int64) * 4096 + d1
    assert np.unique(key).size == key.size
    assert s1.min() >= 0 and s1.max() < 4096 and d1.max() < 4096


def test_rmat_prefix_property():
    """The edge set is the first e distinct valid pairs in attempt order, so a
    smaller e yields a prefix of a larger one."""
    s1, d1 = F.rmat_edges(3, 1000, 3000, 0.57, 0.19, 0.19)
    s2, d2 = F.rmat_edges(3, 1000, 9000, 0.57, 0.19, 0.19)
    assert np.array_equal(s1, s2[:3000]) and np.array_equal(d1, d2[:3000])


@pytest.mark.parametrize("abc", [(0.57, 0.19, 0.19), (0.65, 0.15, 0.15)])
def test_rmat_quadrant_frequencies(abc):
    """Sparse regime (few duplicates): per-level quadrant frequencies match
    (a, b, c, d) within 5 binomial standard deviations."""
    a, b, c = abc
    scale, e = 20, 20000
    s, d = F.rmat_edges(11, 1 << scale, e, a, b, c)
    probs = np.array([a, b, c, 1 - a - b - c])
    for lv in range(scale):
        bit = scale - 1 - lv
        q = ((s >> bit) & 1) * 2 + ((d >> bit) & 1)
        cnt = np.bincount(q, minlength=4)
        sd = np.sqrt(e * probs * (1 - probs))
        assert (np.abs(cnt - e * probs) < 5 * sd + 2).all(), (lv, cnt, e * probs)


def test_features_uniform():
    x = F.features(5, F.UNIFORM, 0, 2000, 64)
    assert x.dtype == np.float32 and x.shape == (2000, 64)
    assert x.min() >= -1.0 and x.max() < 1.0
    # exact multiples of 2^-23
    assert np.all(np.round(x.astype(np.float64) * 2**23) == x.astype(np.float64) * 2**23)
    n = x.size
    assert abs(x.mean()) < 5 * np.sqrt(1 / 3 / n)
    assert abs(x.var() - 1 / 3) < 5 * np.sqrt(4 / 45 / n)
    # rows are keyed by vertex id: a sub-range equals the slice
    y = F.features(5, F.UNIFORM, 100, 300, 64)
    assert np.array_equal(x[100:300], y)
    ids = np.array([7, 1999, 0, 42], np.int64)
    assert np.array_equal(F.features_rows(5, F.UNIFORM, ids, 64), x[ids])


def test_features_normal():
    x = F.features(6, F.NORMAL, 0, 4000, 64).astype(np.float64)
    n = x.size
    assert abs(x.mean()) < 5 / np.sqrt(n)
    assert abs(x.var() - 1.0) < 5 * np.sqrt(2 / n)
    # fourth moment of a standard normal is 3
    assert abs((x**4).mean() - 3.0) < 0.2


@pytest.mark.parametrize("dtype", [F.BF16, F.F16])
def test_features_16bit_are_rne_of_fp32(dtype):
    import torch
    x = F.features(9, F.NORMAL, 0, 500, 32)
    y = F.features(9, F.NORMAL, 0, 500, 32, dtype)
    if dtype == F.F16:
        ref = x.astype(np.float16).view(np.uint16)            # numpy: round to nearest even
    else:
        ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(y, ref)


@pytest.mark.filterwarnings("ignore:overflow encountered")
def test_round16_ties_and_specials():
    import torch
    vals = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, 1.0 + 2**-11, 1.0 + 3 * 2**-11,
                     65504.0, 65519.0, 65520.0, 2**-24, 2**-25, 3 * 2**-25, 6e-8, -0.0,
                     1e-40, -3.5e38], np.float32)
    assert np.array_equal(F.round16(vals, F.F16), vals.astype(np.float16).view(np.uint16))
    bref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(F.round16(vals, F.BF16), bref)


def test_weights_xavier():
    W = F.weights(1, 1, 64, 128, fan_in=128, fan_out=64)
    a = np.sqrt(6 / (128 + 64))
    assert np.abs(W).max() <= a
    n = W.size
    assert abs(W.mean()) < 5 * a * np.sqrt(1 / 3 / n)
    assert abs(W.var() - a * a / 3) < 5 * a * a * np.sqrt(4 / 45 / n)
    W2 = F.weights(1, 2, 64, 128, fan_in=128, fan_out=64)
    assert not np.array_equal(W, W2)
    b = F.bias(1, 1, 64, 128)
    assert np.abs(b).max() <= 1 / np.sqrt(128)


def test_random_ids_is_permutation():
    p = F.random_ids(5, 10000)
    assert np.array_equal(np.sort(p), np.arange(10000))
    assert (p != np.arange(10000)).mean() > 0.99


def test_workload_params_shapes():
    w = WL.SAGE_RMAT_4K
    p = WL.layer_params(w, 1)
    assert p.W.shape == (64, 128) and p.weight_cat().shape == (64, 128)
    p2 = WL.layer_params(WL.GCN_RMAT_1M, 2)
    assert p2.W.shape == (64, 128) and p2.weight_cat().shape == (128, 64)
    p3 = WL.layer_params(WL.SAGE_FANOUT_RMAT_100M, 3)
    assert p3.weight_cat().shape == (256, 344)
    # bf16 workloads carry weights that are exactly bf16 values
    bits = p3.W.view(np.uint32)
    assert (bits & 0xFFFF).max() == 0
