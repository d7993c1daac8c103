"""The shared input generator: numpy and torch views agree bit for bit, and
the distributions have the stated moments -- CPU only."""
import numpy as np
import torch

import datagen as g


def test_hash_reference_values():
    # lowbias32 of small words, evaluated with Python integers
    for x in [0, 1, 2, 0xDEADBEEF, 0xFFFFFFFF]:
        assert int(g.hash32(np.array([x], dtype=np.uint64))[0]) == g._hash32_int(x)
        assert int(g.hash32(torch.tensor([x], dtype=torch.int64))[0]) == g._hash32_int(x)
    assert g._hash32_int(0) == 0


def test_numpy_and_torch_agree():
    w = g.Workload("t", 2, 3, 40, 300, decay=50.0, seed=9)
    assert np.array_equal(g.filters_np(w), g.filters_torch(w, "cpu").numpy())
    assert np.array_equal(g.y_np(w), g.y_torch(w, "cpu").numpy())
    assert np.array_equal(g.x_np(w), g.x_torch(w, "cpu").numpy())
    sub = g.y_np(w, t_idx=[5, 299], m_idx=[1], b_idx=[2], d_idx=[0, 39])
    full = g.y_np(w)
    assert np.array_equal(sub, full[[5, 299]][:, [1]][:, :, [2]][..., [0, 39]])


def test_model_weights_and_noise():
    """The synthetic model's weights and noise: numpy and torch views agree bit
    for bit, the streams are distinct, the scales are the stated ones, and the
    lag-limited filter view is a prefix of the full one."""
    w = g.Workload("m", 2, 3, 16, 300, decay=50.0, seed=4)
    a, b = g.mlp_weights_np(w), g.mlp_weights_torch(w, "cpu")
    assert [x.shape for x in a] == [(2, 32, 16), (2, 32), (2, 16, 32), (2, 16)]
    assert all(np.array_equal(x, y.numpy()) for x, y in zip(a, b))
    assert np.array_equal(g.noise_np(w), g.noise_torch(w, "cpu").numpy())
    assert np.array_equal(g.noise_np(w, 7, 20), g.noise_np(w)[7:20])
    s_up, s_down, s_b = g.mlp_scales(w)
    assert s_up == 1 / 4.0
    norm = np.sqrt(np.sum(np.exp(-2 * np.arange(300) / 50.0)))
    assert abs(s_down - 1 / (2 * norm * np.sqrt(32))) < 1e-15
    big = g.Workload("mb", 1, 1, 256, 16, decay=5.0, seed=1)
    wu = g.mlp_weights_np(big)[0]
    assert abs(wu.std() * np.sqrt(256) - 1) < 0.01
    assert not np.array_equal(a[1][0, :16], a[3][0])          # distinct streams
    assert np.array_equal(g.filters_np(w, lags=37), g.filters_np(w)[:, :, :37])
    assert np.array_equal(g.rho_np(w), g.rho_torch(w, "cpu").numpy())
    assert np.array_equal(g.rho_torch(w, "cpu", 40, 90).numpy(), g.rho_np(w)[40:90])
    assert np.array_equal(g.rho_np(w, t_idx=[3, 7], b_idx=[1]), g.rho_np(w)[[3, 7]][:, :, [1]])


def test_moments_and_ranges():
    n = np.arange(1 << 20, dtype=np.uint64)
    u = g.uniform(n, 1, 1)
    assert 0.0 <= u.min() and u.max() < 1.0 and abs(u.mean() - 0.5) < 2e-3
    z = g.normal(n, 1, 2)
    assert abs(z.mean()) < 5e-3 and abs(z.std() - 1.0) < 5e-3
    assert np.abs(z).max() <= 2 * np.sqrt(3.0)
    v = g.small_int(n, 1, 3, r=3)
    assert set(np.unique(v)) == {-3.0, -2.0, -1.0, 0.0, 1.0, 2.0, 3.0}


def test_large_index_words_differ_by_high_bits():
    lo = np.array([5], dtype=np.uint64)
    hi = lo + np.uint64(1 << 32)
    assert g.words(lo, 1, 1)[0] != g.words(hi, 1, 1)[0]


def test_workloads():
    assert [w.name for w in g.WORKLOADS.values()] == [
        "m1b1d16l1k", "m1b8d768l8k", "m18b4d768l32k", "m18b1d1024l128k", "m32b16d2048l16k"]
    w = g.WORKLOADS["m1b8d768l8k"]
    cols = g.sample_columns(w, 64)
    assert len(cols) == 64 and cols[:, 2].max() < w.D
