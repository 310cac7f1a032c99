"""The seeded input generator: distribution, determinism, shapes (CPU only)."""
import math

import numpy as np
import pytest
import torch

from paper_2204_05436_amd import configs, workload as W


@pytest.mark.parametrize("N,alpha", [(1, 1.1), (2, 1.05), (7, 1.2), (50, 1.1), (1000, 0.8), (300, 1.0)])
def test_zipf_matches_pmf(N, alpha):
    rng = np.random.default_rng(5)
    n = 400_000
    k = W.zipf_ranks(rng, n, N, alpha)
    assert k.min() >= 1 and k.max() <= N
    p = np.arange(1, N + 1, dtype=np.float64) ** -alpha
    p /= p.sum()
    emp = np.bincount(k, minlength=N + 1)[1:] / n
    # each frequency within 6 standard errors of its probability
    se = np.sqrt(p * (1 - p) / n) + 1e-12
    assert np.all(np.abs(emp - p) <= 6 * se + 1e-9)


def test_affine_map_is_bijection():
    w = configs.WORKLOADS["tiny"]
    for N in [1, 2, 7, 97, 1000]:
        r = W.zipf_rows(w, 0, N, np.arange(1, N + 1))
        assert sorted(r.tolist()) == list(range(N))


@pytest.mark.parametrize("name", configs.ORDER)
def test_batch_shapes_and_determinism(name):
    w = configs.WORKLOADS[name]
    if name == "dlrm-large":
        w = configs.scaled(w, batch=512)
    rows = W.table_rows(w)
    a = W.make_batch(w, rows, 3)
    b = W.make_batch(w, rows, 3)
    c = W.make_batch(w, rows, 4)
    assert (a.rows == b.rows).all() and (a.bag_ptr == b.bag_ptr).all()
    assert not np.array_equal(a.rows, c.rows)
    assert a.n_bags == w.batch * w.bags_per_sample
    lens = np.diff(a.bag_ptr)
    if w.bag_len_poisson:
        lo, hi = w.bag_len_clip
        assert lens.min() >= lo and lens.max() <= hi
        assert abs(lens.mean() - w.bag_len_poisson) < 1.0
    else:
        assert (lens == 1).all()
    table = np.repeat(np.arange(a.n_bags) % w.n_tables, lens)
    assert (a.rows < rows[table]).all()


def test_tbsm_locality():
    w = configs.WORKLOADS["tbsm"]
    rows = W.table_rows(w)
    b = W.make_batch(w, rows, 0)
    r = b.rows.reshape(w.batch, w.steps, w.n_tables)
    same = (r[:, 1:, :] == r[:, :-1, :]).mean()
    assert 0.68 < same < 0.80   # 70% copies plus chance equality of fresh draws


def test_row_counts():
    w = configs.WORKLOADS["dlrm-large"]
    rows = W.table_rows(w)
    assert len(rows) == 26 and rows.min() >= 100 and rows.max() <= 40_000_000
    assert (W.table_rows(w) == rows).all()
    assert configs.WORKLOADS["dlrm-large"].k_cap(int(rows.sum())) == 16_777_216
    assert configs.WORKLOADS["tiny"].k_cap(80_000) == 800
    assert configs.WORKLOADS["tbsm"].k_cap(1_110_000) == 11_100
    assert configs.WORKLOADS["multi-hot"].k_cap(40_000_000) == 800_000
    assert configs.WORKLOADS["dlrm-small"].k_cap(1) == 8_388_608


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_weights_numpy_equals_torch(dtype):
    w = configs.scaled(configs.WORKLOADS["tiny"], dtype=dtype, dim=24)
    n = 5000
    a = np.empty((n, w.dim), np.float32 if dtype == "f32" else np.uint16)
    W.fill_weights_np(w, a, row0=123_456_789, chunk_rows=777)
    t = torch.empty((n, w.dim), dtype=torch.float32 if dtype == "f32" else torch.int16)
    W.fill_weights_torch(w, t, "cpu", row0=123_456_789, chunk_rows=1000)
    assert (t.numpy().view(a.dtype) == a).all()
    # counter-based: a row is the same whichever chunk produced it
    assert (W.weight_rows(w, np.array([123_456_789 + 17])) == a[17]).all()
    f = a if dtype == "f32" else (a.astype(np.uint32) << 16).view(np.float32)
    assert f.min() >= -0.0501 and f.max() < 0.0501 and abs(float(f.mean())) < 2e-3
    # large element indices (beyond 2^32) take the high word into account
    big = W.weight_values_f32(w, np.array([5, 5 + (1 << 32)], np.uint64))
    assert big[0] != big[1]


def test_dy_and_dense():
    w = configs.WORKLOADS["dlrm-small"]
    d = W.make_dy(w, 0, 100)
    assert d.shape == (100, 16) and d.dtype == np.float32 and abs(float(d.std()) - 1) < 0.1
    assert W.make_dense(w, 0).shape == (4096, 13)
