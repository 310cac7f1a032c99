"""Python marshalling for the C oracle (hotline_oracle.c) -- TEST INFRASTRUCTURE.

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It shares no code with the HIP library and never calls
it.  Every function takes and returns numpy arrays; the arithmetic is all in
the C file.

``mc_*`` wrap cpu_segregation_mc.c, which is not the oracle: a multi-core
(OpenMP) classify + partition that the benchmark reports as a labelled CPU
baseline, checked bit for bit against the oracle by the tests.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hotline_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_MC_SRC = os.path.join(_HERE, "cpu_segregation_mc.c")
_MC_LIB = os.path.join(_HERE, "libcpuseg_mc.so")
F32, BF16 = 0, 1

_lib = None


# gcc's AddressSanitizer and UndefinedBehaviorSanitizer, any finding fatal
SAN_FLAGS = ["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all"]


def build(force: bool = False, out: str | None = None, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (single-threaded, fp64, no FMA contraction).
    With ``sanitize`` the copy at ``out`` carries gcc's ASan and UBSan checks; a
    process that loads it preloads gcc's libasan (``gcc -print-file-name=libasan.so``)."""
    lib_path = out or _LIB
    if force or sanitize or not os.path.exists(lib_path) or os.path.getmtime(lib_path) < os.path.getmtime(_SRC):
        tmp = lib_path + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c99",
                               "-Wall", "-Wextra", *(SAN_FLAGS if sanitize else ()),
                               "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, lib_path)
    if out is None and not sanitize:
        build_mc(force)
    return lib_path


def build_mc(force: bool = False) -> str:
    """Compile the multi-core CPU segregation baseline (OpenMP; not the oracle)."""
    if force or not os.path.exists(_MC_LIB) or os.path.getmtime(_MC_LIB) < os.path.getmtime(_MC_SRC):
        tmp = _MC_LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-std=c99", "-Wall", "-Wextra", "-shared", "-fPIC",
                               _MC_SRC, "-o", tmp])
        os.replace(tmp, _MC_LIB)
    return _MC_LIB


def lib():
    global _lib
    if _lib is None:
        L = C.CDLL(build())
        P = C.c_void_p
        i32, i64, u32, u64, f32 = C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_float
        sig = {
            "ho_gids": (C.c_int, [i32, P, P, P, i64, P]),
            "ho_count": (C.c_int, [u64, P, i64, P]),
            "ho_topk": (i64, [u64, P, u64, P]),
            "ho_classify": (None, [P, i64, P, P, i32, i32, P]),
            "ho_partition": (i32, [P, i32, P, P]),
            "ho_remap": (None, [P, i64, P, i64, P]),
            "ho_cold_plan": (i64, [P, P, P, P, i32, i32, u32, P]),
            "ho_gather": (None, [P, u64, P, i64, P]),
            "ho_scatter": (None, [P, u64, P, i64, P]),
            "ho_embbag_fwd": (C.c_int, [i32, i32, P, u32, i64, P, i64, P, P, P, i32, i32, P, P]),
            "ho_embbag_fwd_flat": (None, [i32, i32, P, P, P, i64, P]),
            "ho_embbag_bwd_sgd": (i64, [i32, i32, P, u32, i64, P, i64, P, P, P, i32, i32, P, f32,
                                        P, P]),
            "ho_embbag_bwd_sgd_flat": (None, [i32, i32, P, P, P, i64, P, f32]),
            "ho_round_bf16": (C.c_uint16, [C.c_double]),
            "ho_migrate": (i64, [u64, P, i64, P, P, i64, P, P]),
            "ho_mix32": (u32, [u32]),
            "ho_eal_init": (None, [i64, i32, P, P]),
            "ho_eal_access": (None, [i64, i32, P, P, P, i64]),
            "ho_eal_hot": (i64, [i64, i32, P, P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


_mc = None


def mc_lib():
    """The multi-core segregation baseline (cpu_segregation_mc.c)."""
    global _mc
    if _mc is None:
        L = C.CDLL(build_mc())
        P = C.c_void_p
        L.mc_hot_bitmap.restype = C.c_int
        L.mc_hot_bitmap.argtypes = [P, C.c_int64, C.c_uint64, P]
        L.mc_segregate.restype = C.c_int32
        L.mc_segregate.argtypes = [C.c_int32, P, P, P, C.c_int32, C.c_int32, P, C.c_int32, P, P, P]
        _mc = L
    return _mc


def mc_hot_bitmap(hot_ids, n_rows):
    hot_ids = _c(hot_ids, np.uint32)
    bm = np.empty((int(n_rows) + 63) // 64, dtype=np.uint64)
    rc = mc_lib().mc_hot_bitmap(_p(hot_ids), len(hot_ids), int(n_rows), _p(bm))
    return bm, rc


def mc_segregate(rows_per_table, rows, bag_ptr, n_samples, bps, bm, n_threads, out=None):
    """(flags, pop, nonpop) of the multi-core segregation; ``out`` may hold
    preallocated (flags, pop, nonpop) arrays of n_samples entries."""
    rpt = _c(rows_per_table, np.uint32)
    rows = _c(rows, np.uint32)
    bag_ptr = _c(bag_ptr, np.int32)
    if out is None:
        out = (np.empty(n_samples, dtype=np.uint8), np.empty(n_samples, dtype=np.int32),
               np.empty(n_samples, dtype=np.int32))
    flags, pop, nonpop = out
    npop = mc_lib().mc_segregate(len(rpt), _p(rpt), _p(rows), _p(bag_ptr), n_samples, bps, _p(bm),
                                 n_threads, _p(flags), _p(pop), _p(nonpop))
    if npop < 0:
        raise ValueError("mc_segregate: bad argument")
    return flags[:n_samples], pop[:npop], nonpop[: n_samples - npop]


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def dtype_code(dtype: str) -> int:
    return F32 if dtype == "f32" else BF16


def storage_np(dtype: str):
    return np.float32 if dtype == "f32" else np.uint16


# ---------------------------------------------------------------------------- steps
def gids(rows_per_table, rows, bag_ptr):
    rpt = _c(rows_per_table, np.uint32)
    rows = _c(rows, np.uint32)
    bag_ptr = _c(bag_ptr, np.int32)
    out = np.empty(len(rows), dtype=np.uint32)
    rc = lib().ho_gids(len(rpt), _p(rpt), _p(rows), _p(bag_ptr), len(bag_ptr) - 1, _p(out))
    return out, rc


def count(n_rows, gid_batches, counts=None):
    counts = np.zeros(n_rows, dtype=np.uint32) if counts is None else counts
    rc = 0
    for g in gid_batches:
        g = _c(g, np.uint32)
        rc |= lib().ho_count(n_rows, _p(g), len(g), _p(counts))
    return counts, rc


def topk(counts, k):
    counts = _c(counts, np.uint32)
    out = np.empty(max(1, min(int(k), len(counts))), dtype=np.uint32)
    nh = lib().ho_topk(len(counts), _p(counts), int(k), _p(out))
    return out[:nh].copy()


def classify(hot_ids, gids_, bag_ptr, n_samples, bps):
    hot_ids = _c(hot_ids, np.uint32)
    gids_ = _c(gids_, np.uint32)
    bag_ptr = _c(bag_ptr, np.int32)
    flags = np.empty(n_samples, dtype=np.uint8)
    lib().ho_classify(_p(hot_ids), len(hot_ids), _p(gids_), _p(bag_ptr), n_samples, bps, _p(flags))
    return flags


def partition(flags):
    flags = _c(flags, np.uint8)
    n = len(flags)
    pop = np.empty(n, dtype=np.int32)
    nonpop = np.empty(n, dtype=np.int32)
    npop = lib().ho_partition(_p(flags), n, _p(pop), _p(nonpop))
    return pop[:npop].copy(), nonpop[: n - npop].copy()


def remap(hot_ids, gids_):
    hot_ids = _c(hot_ids, np.uint32)
    gids_ = _c(gids_, np.uint32)
    codes = np.empty(len(gids_), dtype=np.int32)
    lib().ho_remap(_p(hot_ids), len(hot_ids), _p(gids_), len(gids_), _p(codes))
    return codes


def cold_plan(gids_, codes, bag_ptr, sel, n_sel, bps, k_cap):
    """Returns (cold_ids, codes_rewritten); the input codes are not modified."""
    gids_ = _c(gids_, np.uint32)
    codes = np.array(codes, dtype=np.int32, copy=True)
    bag_ptr = _c(bag_ptr, np.int32)
    sel = None if sel is None else _c(sel, np.int32)
    cold = np.empty(max(1, len(codes)), dtype=np.uint32)
    n = lib().ho_cold_plan(_p(gids_), _p(codes), _p(bag_ptr), _p(sel), n_sel, bps, int(k_cap), _p(cold))
    return cold[:n].copy(), codes


def gather(table, ids):
    """table: [n_rows, dim] array (any dtype); returns table[ids] via the oracle's row copy."""
    table = np.ascontiguousarray(table)
    ids = _c(ids, np.uint32)
    out = np.empty((len(ids),) + table.shape[1:], dtype=table.dtype)
    rb = table.strides[0]
    lib().ho_gather(_p(table), rb, _p(ids), len(ids), _p(out))
    return out


def scatter(table, ids, rows):
    """table[ids] = rows in place via the oracle's write-back (ids distinct)."""
    assert table.flags.c_contiguous
    ids = _c(ids, np.uint32)
    rows = np.ascontiguousarray(rows, dtype=table.dtype)
    assert rows.shape == (len(ids),) + table.shape[1:]
    lib().ho_scatter(_p(table), table.strides[0], _p(ids), len(ids), _p(rows))


def migrate(old_ids, w_hot_old, new_ids, host):
    """Hot-set migration (re-learning): returns (w_hot_new, n_written_back);
    host ([n_rows, dim], C-contiguous) is updated in place.  w_hot_old holds the
    old set's rows by slot (at least len(old_ids) rows)."""
    assert host.flags.c_contiguous
    old_ids, new_ids = _c(old_ids, np.uint32), _c(new_ids, np.uint32)
    w_hot_old = np.ascontiguousarray(w_hot_old, dtype=host.dtype)
    out = np.empty((len(new_ids),) + host.shape[1:], dtype=host.dtype)
    n = lib().ho_migrate(host.strides[0], _p(old_ids), len(old_ids), _p(w_hot_old), _p(new_ids), len(new_ids),
                         _p(out), _p(host))
    return out, int(n)


class EAL:
    """The SRRIP access logger (oracle): n_sets x ways (id, RRPV) entries."""

    def __init__(self, n_sets: int, ways: int):
        self.n_sets, self.ways = int(n_sets), int(ways)
        self.tag = np.empty(self.n_sets * self.ways, np.uint32)
        self.rrpv = np.empty(self.n_sets * self.ways, np.uint8)
        lib().ho_eal_init(self.n_sets, self.ways, _p(self.tag), _p(self.rrpv))

    def access(self, gids_):
        g = _c(gids_, np.uint32)
        lib().ho_eal_access(self.n_sets, self.ways, _p(self.tag), _p(self.rrpv), _p(g), len(g))

    def hot(self):
        out = np.empty(max(1, self.tag.size), np.uint32)
        n = lib().ho_eal_hot(self.n_sets, self.ways, _p(self.tag), _p(out))
        return out[:n].copy()


def mix32(x: int) -> int:
    return int(lib().ho_mix32(int(x) & 0xFFFFFFFF))


def gather_ptr(table_ptr: int, row_bytes: int, ids, dim: int, np_dtype):
    ids = _c(ids, np.uint32)
    out = np.empty((len(ids), dim), dtype=np_dtype)
    lib().ho_gather(C.c_void_p(table_ptr), row_bytes, _p(ids), len(ids), _p(out))
    return out


def embbag_fwd(dtype, w_hot, k_cap, staging, codes, bag_ptr, sel, n_sel, bps, n_bags_total,
               want_scale=False):
    dim = w_hot.shape[1]
    w_hot = np.ascontiguousarray(w_hot)
    staging = np.ascontiguousarray(staging) if staging is not None else np.zeros((0, dim), w_hot.dtype)
    codes = _c(codes, np.int32)
    bag_ptr = _c(bag_ptr, np.int32)
    sel = None if sel is None else _c(sel, np.int32)
    out = np.zeros((n_bags_total, dim), dtype=np.float32)
    scale = np.zeros((n_bags_total, dim), dtype=np.float64) if want_scale else None
    rc = lib().ho_embbag_fwd(dim, dtype_code(dtype), _p(w_hot), int(k_cap), len(w_hot), _p(staging),
                             len(staging), _p(codes), _p(bag_ptr), _p(sel), n_sel, bps, _p(out),
                             _p(scale))
    return out, scale, rc


def embbag_fwd_flat(dtype, table, gids_, bag_ptr):
    table = np.ascontiguousarray(table)
    gids_ = _c(gids_, np.uint32)
    bag_ptr = _c(bag_ptr, np.int32)
    out = np.empty((len(bag_ptr) - 1, table.shape[1]), dtype=np.float32)
    lib().ho_embbag_fwd_flat(table.shape[1], dtype_code(dtype), _p(table), _p(gids_), _p(bag_ptr),
                             len(bag_ptr) - 1, _p(out))
    return out


def embbag_bwd_sgd(dtype, w_hot, k_cap, staging, codes, bag_ptr, sel, n_sel, bps, dY, lr,
                   want_scale=False):
    """Updates w_hot / staging IN PLACE.  Returns (uniq_codes, scale[n_u, dim] or None, rc)."""
    dim = w_hot.shape[1]
    assert w_hot.flags.c_contiguous and (staging is None or staging.flags.c_contiguous)
    if staging is None:
        staging = np.zeros((0, dim), w_hot.dtype)
    codes = _c(codes, np.int32)
    bag_ptr = _c(bag_ptr, np.int32)
    sel = None if sel is None else _c(sel, np.int32)
    dY = _c(dY, np.float32)
    m = int(len(codes))
    uniq = np.empty(max(1, m), dtype=np.int32)
    scale = np.empty((max(1, m), dim), dtype=np.float64) if want_scale else None
    nu = lib().ho_embbag_bwd_sgd(dim, dtype_code(dtype), _p(w_hot), int(k_cap), len(w_hot),
                                 _p(staging), len(staging), _p(codes), _p(bag_ptr), _p(sel), n_sel,
                                 bps, _p(dY), float(lr), _p(uniq), _p(scale))
    if nu < 0:
        return None, None, int(nu)
    return uniq[:nu].copy(), (scale[:nu].copy() if want_scale else None), 0


def embbag_bwd_sgd_flat(dtype, table, gids_, bag_ptr, dY, lr):
    assert table.flags.c_contiguous
    gids_ = _c(gids_, np.uint32)
    bag_ptr = _c(bag_ptr, np.int32)
    dY = _c(dY, np.float32)
    lib().ho_embbag_bwd_sgd_flat(table.shape[1], dtype_code(dtype), _p(table), _p(gids_), _p(bag_ptr),
                                 len(bag_ptr) - 1, _p(dY), float(lr))


def round_bf16(x: float) -> int:
    return int(lib().ho_round_bf16(float(x)))


# ---------------------------------------------------------------------------- whole path
def run_path(w, rows_per_table, prof_batches, batch, dY, table, k=None, writeback=False):
    """Every step of the hot path for one measured mini-batch, in the paper's order:
    profile (count + select), classify, partition, remap, cold plan + gather, forward
    over both mu-batches, one coalesced SGD step [, write-back of the updated cold
    rows into a copy of the table: key "table_new"].  `table` is the full host table
    [n_rows, dim] (float32 or uint16 bf16 bits); it is not modified.
    Returns a dict of every intermediate and final result."""
    n_rows = int(np.sum(rows_per_table, dtype=np.int64))
    k_cap = w.k_cap(n_rows) if k is None else int(k)
    counts = np.zeros(n_rows, dtype=np.uint32)
    for pb in prof_batches:
        g, _ = gids(rows_per_table, pb.rows, pb.bag_ptr)
        count(n_rows, [g], counts)
    hot = topk(counts, k_cap)
    g, rc_g = gids(rows_per_table, batch.rows, batch.bag_ptr)
    B, bps = batch.n_samples, batch.bags_per_sample
    flags = classify(hot, g, batch.bag_ptr, B, bps)
    pop, nonpop = partition(flags)
    codes0 = remap(hot, g)
    cold, codes = cold_plan(g, codes0, batch.bag_ptr, nonpop, len(nonpop), bps, k_cap)
    w_hot = gather(table, hot)
    stg = gather(table, cold)
    out, scale_f, rc1 = embbag_fwd(w.dtype, w_hot, k_cap, stg, codes, batch.bag_ptr, pop, len(pop),
                                    bps, batch.n_bags, want_scale=True)
    out2, scale2, rc2 = embbag_fwd(w.dtype, w_hot, k_cap, stg, codes, batch.bag_ptr, nonpop,
                                    len(nonpop), bps, batch.n_bags, want_scale=True)
    sel_np = np.zeros(batch.n_bags, dtype=bool)
    for s in nonpop:
        sel_np[s * bps:(s + 1) * bps] = True
    out[sel_np] = out2[sel_np]
    scale_f[sel_np] = scale2[sel_np]
    w_hot_new = w_hot.copy()
    stg_new = stg.copy()
    uniq, scale_b, rc3 = embbag_bwd_sgd(w.dtype, w_hot_new, k_cap, stg_new, codes, batch.bag_ptr,
                                        None, B, bps, dY, w.lr, want_scale=True)
    r = dict(n_rows=n_rows, k_cap=k_cap, counts=counts, hot=hot, gids=g, flags=flags, pop=pop,
             nonpop=nonpop, codes_remap=codes0, cold=cold, codes=codes, w_hot=w_hot, staging=stg,
             out=out, out_scale=scale_f, w_hot_new=w_hot_new, staging_new=stg_new, uniq=uniq,
             upd_scale=scale_b, rc=(rc_g, rc1, rc2, rc3))
    if writeback:
        r["table_new"] = np.array(table, copy=True)
        scatter(r["table_new"], cold, stg_new)
    return r
