"""The multi-core CPU segregation baseline (oracle/cpu_segregation_mc.c, the
classify + partition on the host's cores that Sec. III measures) against the
oracle's ho_gids + ho_classify + ho_partition, bit for bit, at several thread
counts.  CPU only."""
import numpy as np
import pytest

import oracle as O


def _case(seed, n_tables, steps, n_samples, max_len, hot_frac, bad_rows=0):
    rng = np.random.default_rng(seed)
    rpt = rng.integers(1, 400, n_tables).astype(np.uint32)
    bps = n_tables * steps
    lens = rng.integers(0 if max_len > 1 else 1, max_len + 1, n_samples * bps)
    bag_ptr = np.zeros(n_samples * bps + 1, dtype=np.int32)
    bag_ptr[1:] = np.cumsum(lens)
    table_of = np.repeat(np.arange(n_samples * bps) % n_tables, lens)
    # skewed rows: most lookups fall on each table's first few rows
    rows = np.minimum(rng.zipf(1.3, len(table_of)) - 1, rpt[table_of] - 1).astype(np.uint32)
    if bad_rows:
        at = rng.choice(len(rows), min(bad_rows, len(rows)), replace=False)
        rows[at] = rpt[table_of[at]] + rng.integers(0, 5, len(at)).astype(np.uint32)
    n_rows = int(rpt.sum())
    k = int(round(hot_frac * n_rows))
    # the hot set: the k most-accessed rows (ties by id), as a learning phase picks them
    base = np.concatenate([[0], np.cumsum(rpt.astype(np.int64))[:-1]])
    ok = rows < rpt[table_of]
    cnt = np.bincount(base[table_of[ok]] + rows[ok], minlength=n_rows)
    hot = np.sort(np.lexsort((np.arange(n_rows), -cnt))[:k]).astype(np.uint32)
    return rpt, rows, bag_ptr, bps, hot, n_rows


def _oracle(rpt, rows, bag_ptr, n_samples, bps, hot):
    g, _ = O.gids(rpt, rows, bag_ptr)
    flags = O.classify(hot, g, bag_ptr, n_samples, bps)
    pop, nonpop = O.partition(flags)
    return flags, pop, nonpop


@pytest.mark.parametrize("threads", [1, 2, 3, 7, 16])
@pytest.mark.parametrize("shape", [
    dict(n_tables=5, steps=1, n_samples=1000, max_len=1, hot_frac=0.05),     # one-hot
    dict(n_tables=3, steps=4, n_samples=333, max_len=4, hot_frac=0.2),       # multi-hot, empty bags
    dict(n_tables=2, steps=1, n_samples=5, max_len=3, hot_frac=0.5),         # fewer samples than threads
    dict(n_tables=4, steps=1, n_samples=700, max_len=2, hot_frac=0.1, bad_rows=25),  # rows outside tables
    dict(n_tables=3, steps=1, n_samples=0, max_len=1, hot_frac=0.1),         # empty batch
    dict(n_tables=3, steps=2, n_samples=200, max_len=3, hot_frac=0.0),       # no hot row
    dict(n_tables=3, steps=2, n_samples=200, max_len=3, hot_frac=1.0),       # every row hot
])
def test_matches_oracle(shape, threads):
    rpt, rows, bag_ptr, bps, hot, n_rows = _case(11 + threads, **shape)
    n = shape["n_samples"]
    bm, rc = O.mc_hot_bitmap(hot, n_rows)
    assert rc == 0
    f, p, q = O.mc_segregate(rpt, rows, bag_ptr, n, bps, bm, threads)
    fo, po, qo = _oracle(rpt, rows, bag_ptr, n, bps, hot)
    assert np.array_equal(f, fo)
    assert np.array_equal(p, po)
    assert np.array_equal(q, qo)


def test_hot_bitmap():
    hot = np.array([0, 5, 63, 64, 130, 199], dtype=np.uint32)
    bm, rc = O.mc_hot_bitmap(hot, 200)
    assert rc == 0 and len(bm) == 4
    bits = np.unpackbits(bm.view(np.uint8), bitorder="little")[:200]
    assert np.array_equal(np.flatnonzero(bits), hot)
    bm, rc = O.mc_hot_bitmap(np.array([3, 200], dtype=np.uint32), 200)   # an id past the rows
    assert rc == 2
    assert np.array_equal(np.flatnonzero(np.unpackbits(bm.view(np.uint8), bitorder="little")[:200]), [3])


def test_bad_arguments():
    bm, _ = O.mc_hot_bitmap(np.zeros(0, dtype=np.uint32), 10)
    with pytest.raises(ValueError):
        O.mc_segregate(np.zeros(0, dtype=np.uint32), np.zeros(0, dtype=np.uint32), np.zeros(1, dtype=np.int32),
                       0, 1, bm, 4)
