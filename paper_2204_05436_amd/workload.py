"""Seeded synthetic inputs for the hot path (shared by the kernels' tests, the
oracle's tests and the benchmark).

This module only draws inputs: table sizes, per-lookup table-local row ids in
CSR bag layout, gradients, dense features and the initial weight values.  It
performs none of the method's own arithmetic (no global-id formation, no
counting, selection, classification or pooling).

Index distribution: per table, rank k in 1..N has probability proportional to
k^-alpha (Zipf), sampled with the rejection-inversion method of Hoermann and
Derflinger (ACM TOMACS 6(3), 1996), written here from that description.
Ranks are mapped to rows through a seeded affine bijection row = (a*(k-1)+c)
mod N (gcd(a, N) = 1), so popular rows are scattered over the table the way
hashed categorical ids are.

Batch layout (sample-major CSR): bag index = (b*steps + s)*n_tables + t, sample
b owns bags [b*bps, (b+1)*bps), bag_ptr[n_bags+1] indexes the rows array.

Weights come from a counter-based integer hash of (seed, element index), so any
row can be regenerated independently, on the CPU with numpy or on a GPU with
torch, bit-identically.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

from .configs import Workload

# purposes for the seed sequence
_P_ROWS, _P_IDX, _P_LEN, _P_PERM, _P_DY, _P_DENSE = 1, 2, 3, 5, 6, 7


def _rng(*words) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(x) for x in words])))


# ----------------------------------------------------------------------------- tables
def table_rows(w: Workload) -> np.ndarray:
    """Rows per table (uint32).  Log-uniform tables: round(exp(U(ln lo, ln hi)))."""
    if w.rows_fixed:
        rows = np.asarray(w.rows_fixed, dtype=np.int64)
    else:
        lo, hi = w.rows_loguniform
        u = _rng(w.seed, _P_ROWS).uniform(math.log(lo), math.log(hi), size=w.n_tables)
        rows = np.maximum(1, np.rint(np.exp(u))).astype(np.int64)
    assert rows.sum() < 2**32 - 1
    return rows.astype(np.uint32)


def _affine(w: Workload, t: int, n: int, phase: int = 0):
    # phase > 0: another bijection, as if user behaviour had shifted (the skew
    # evolves, Sec. III challenge 3); phase 0 is the stream's own
    r = _rng(w.seed, _P_PERM, t) if phase == 0 else _rng(w.seed, _P_PERM, t, phase)
    if n == 1:
        return 1, 0
    while True:
        a = int(r.integers(1, n))
        if math.gcd(a, n) == 1:
            break
    c = int(r.integers(0, n))
    return a, c


# ----------------------------------------------------------------------------- zipf
def _h1(z):  # log1p(z)/z, continuous at 0
    z = np.asarray(z, dtype=np.float64)
    out = np.ones_like(z)
    big = np.abs(z) > 1e-8
    out[big] = np.log1p(z[big]) / z[big]
    out[~big] = 1.0 - z[~big] / 2.0 + z[~big] ** 2 / 3.0
    return out


def _h2(z):  # expm1(z)/z, continuous at 0
    z = np.asarray(z, dtype=np.float64)
    out = np.ones_like(z)
    big = np.abs(z) > 1e-8
    out[big] = np.expm1(z[big]) / z[big]
    out[~big] = 1.0 + z[~big] / 2.0 + z[~big] ** 2 / 6.0
    return out


def zipf_ranks(rng: np.random.Generator, n: int, N: int, alpha: float) -> np.ndarray:
    """n i.i.d. ranks in [1, N] with P(k) proportional to k^-alpha (int64)."""
    if N == 1 or n == 0:
        return np.ones(n, dtype=np.int64)
    s = float(alpha)

    def H(x):  # antiderivative of x^-s with H(1) = 0
        lx = np.log(x)
        return _h2((1.0 - s) * lx) * lx

    def Hinv(y):
        return np.exp(_h1((1.0 - s) * y) * y)

    def h(x):
        return np.exp(-s * np.log(x))

    hx1 = float(H(np.array([1.5]))[0]) - 1.0
    hN = float(H(np.array([N + 0.5]))[0])
    thr = 2.0 - float(Hinv(H(np.array([2.5])) - h(np.array([2.0])))[0])
    out = np.empty(n, dtype=np.int64)
    todo = np.arange(n)
    while todo.size:
        u = hN + rng.random(todo.size) * (hx1 - hN)
        x = Hinv(u)
        k = np.clip(np.floor(x + 0.5), 1, N)
        ok = (k - x <= thr) | (u >= H(k + 0.5) - h(k))
        out[todo[ok]] = k[ok].astype(np.int64)
        todo = todo[~ok]
    return out


def zipf_rows(w: Workload, t: int, N: int, ranks: np.ndarray, phase: int = 0) -> np.ndarray:
    a, c = _affine(w, t, N, phase)
    r = (np.uint64(a) * (ranks.astype(np.uint64) - np.uint64(1)) + np.uint64(c)) % np.uint64(N)
    return r.astype(np.uint32)


# ----------------------------------------------------------------------------- batches
@dataclass
class Batch:
    index: int
    rows: np.ndarray      # uint32 [L]  table-local row id of every lookup
    bag_ptr: np.ndarray   # int32 [n_bags+1]
    n_samples: int
    bags_per_sample: int

    @property
    def n_lookups(self) -> int:
        return int(self.bag_ptr[-1])

    @property
    def n_bags(self) -> int:
        return len(self.bag_ptr) - 1


def make_batch(w: Workload, rows_per_table: np.ndarray, index: int, phase: int = 0) -> Batch:
    """Mini-batch number `index` of the seeded stream (independent of other
    batches); phase > 0 maps the same Zipf ranks to other rows (a drifted
    popularity)."""
    B, T, S = w.batch, w.n_tables, w.steps
    n_bags = B * S * T
    if w.bag_len_poisson > 0:
        assert S == 1
        lo, hi = w.bag_len_clip
        lens = np.clip(_rng(w.seed, _P_LEN, index).poisson(w.bag_len_poisson, size=(B, T)), lo, hi)
        lens = lens.astype(np.int64)
        bag_ptr = np.zeros(n_bags + 1, dtype=np.int64)
        np.cumsum(lens.reshape(-1), out=bag_ptr[1:])
        rows = np.empty(int(bag_ptr[-1]), dtype=np.uint32)
        for t in range(T):
            N = int(rows_per_table[t])
            lt = lens[:, t]
            tot = int(lt.sum())
            ranks = zipf_ranks(_rng(w.seed, _P_IDX, t, index), tot, N, w.alpha)
            starts = bag_ptr[np.arange(B) * T + t]
            excl = np.concatenate([[0], np.cumsum(lt)[:-1]])
            pos = np.repeat(starts - excl, lt) + np.arange(tot)
            rows[pos] = zipf_rows(w, t, N, ranks, phase)
        return Batch(index, rows, bag_ptr.astype(np.int32), B, T)

    rows = np.empty((B, S, T), dtype=np.uint32)
    for t in range(T):
        N = int(rows_per_table[t])
        r = _rng(w.seed, _P_IDX, t, index)
        fresh = zipf_rows(w, t, N, zipf_ranks(r, B * S, N, w.alpha), phase).reshape(B, S)
        if S > 1 and w.repeat_prob > 0:
            coin = r.random((B, S)) < w.repeat_prob
            idx = fresh.copy()
            for s in range(1, S):
                idx[:, s] = np.where(coin[:, s], idx[:, s - 1], fresh[:, s])
            fresh = idx
        rows[:, :, t] = fresh
    bag_ptr = np.arange(n_bags + 1, dtype=np.int32)
    return Batch(index, rows.reshape(-1), bag_ptr, B, S * T)


def make_dy(w: Workload, index: int, n_bags: int) -> np.ndarray:
    """Upstream gradient of the pooled outputs, N(0,1) fp32, [n_bags, dim]."""
    return _rng(w.seed, _P_DY, index).standard_normal((n_bags, w.dim), dtype=np.float32)


def make_dense(w: Workload, index: int) -> np.ndarray:
    """Dense features carried with each sample (not used by the embedding path)."""
    return _rng(w.seed, _P_DENSE, index).standard_normal((w.batch, w.n_dense), dtype=np.float32)


# ----------------------------------------------------------------------------- weights
_M32 = 0xFFFFFFFF
_MUL = 0x45D9F3B
_GOLD = 0x9E3779B9
_SCALE = np.float32(0.05 / 8388608.0)


def _mix32_np(x):
    x = (((x >> np.uint64(16)) ^ x) * np.uint64(_MUL)) & np.uint64(_M32)
    x = (((x >> np.uint64(16)) ^ x) * np.uint64(_MUL)) & np.uint64(_M32)
    return (x >> np.uint64(16)) ^ x


def _weight_seed(w: Workload) -> int:
    return (w.seed * _GOLD + 0x5BD1E995) & _M32


def weight_values_f32(w: Workload, elem_index: np.ndarray) -> np.ndarray:
    """U(-0.05, 0.05) fp32 value of flat element index (row*dim + d)."""
    n = elem_index.astype(np.uint64)
    h = _mix32_np((n >> np.uint64(32)) ^ np.uint64(_weight_seed(w)))
    h = _mix32_np((n & np.uint64(_M32)) ^ h)
    u = (h >> np.uint64(8)).astype(np.int64) - 8388608
    return u.astype(np.float32) * _SCALE


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 bit pattern (finite inputs)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return b.astype(np.uint16)


def weight_rows(w: Workload, flat_rows: np.ndarray) -> np.ndarray:
    """Storage values of the given table rows: float32 [n, dim] or uint16 bf16 bits [n, dim]."""
    flat_rows = np.asarray(flat_rows, dtype=np.uint64)
    idx = flat_rows[:, None] * np.uint64(w.dim) + np.arange(w.dim, dtype=np.uint64)[None, :]
    v = weight_values_f32(w, idx)
    return v if w.dtype == "f32" else f32_to_bf16_bits(v)


def fill_weights_np(w: Workload, out: np.ndarray, row0: int = 0, chunk_rows: int = 1 << 16,
                    threads: int | None = None) -> None:
    """Fill out[r] = weights of table row row0 + r (out: [n, dim] float32 or uint16)."""
    n = out.shape[0]
    threads = threads or min(16, os.cpu_count() or 1)

    def job(a):
        b = min(n, a + chunk_rows)
        out[a:b] = weight_rows(w, np.arange(row0 + a, row0 + b, dtype=np.uint64))

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(job, range(0, n, chunk_rows)))


def fill_weights_torch(w: Workload, out, device, row0: int = 0, chunk_rows: int = 1 << 20) -> None:
    """Same values as fill_weights_np, computed with torch on `device` and copied into
    `out` (a torch tensor [n, dim] float32 or int16, typically in pinned host memory)."""
    import torch

    n = out.shape[0]
    d = torch.arange(w.dim, dtype=torch.int64, device=device)
    seed = _weight_seed(w)

    def mix(x):
        x = (((x >> 16) ^ x) * _MUL) & _M32
        x = (((x >> 16) ^ x) * _MUL) & _M32
        return (x >> 16) ^ x

    scale = torch.tensor(float(_SCALE), dtype=torch.float32, device=device)
    for a in range(0, n, chunk_rows):
        b = min(n, a + chunk_rows)
        r = torch.arange(row0 + a, row0 + b, dtype=torch.int64, device=device)
        e = r[:, None] * w.dim + d[None, :]
        h = mix((e >> 32) ^ seed)
        h = mix((e & _M32) ^ h)
        v = ((h >> 8) - 8388608).to(torch.float32) * scale
        if w.dtype == "f32":
            out[a:b].copy_(v)
        else:
            out[a:b].copy_(v.to(torch.bfloat16).view(torch.int16))
