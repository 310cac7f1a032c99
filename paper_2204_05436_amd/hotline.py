"""Thin ctypes binding of libhotline.so (include/hotline.h): one Python function
per C entry point, same names, argument marshalling only.  Device buffers are
torch tensors (their data_ptr is passed); streams are torch streams.  Raises
ImportError when the HIP library has not been built: there is no fallback."""
from __future__ import annotations

import atexit
import ctypes as C
import itertools
import os
import sys

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# HOTLINE_LIB names another build of the same library (a host-sanitized copy)
LIB_PATH = os.environ.get("HOTLINE_LIB") or os.path.join(_HERE, "libhotline.so")

HL_F32, HL_BF16 = 0, 1
STATUS = {0: "ok", 1: "invalid argument", 2: "out of range", 3: "capacity exceeded", 4: "HIP runtime error",
          5: "unsupported", 6: "device error word set"}
DEVERR = {"OUT_OF_RANGE": 0x1, "BAD_CODE": 0x2, "CAPACITY": 0x4, "BAD_HOTSET": 0x8, "STALL": 0x10,
          "SHAPE": 0x20, "INTERNAL": 0x40}


class HotlineError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn}: {STATUS.get(status, status)} ({status})")
        self.status = status


_lib = None
P, I32, I64, U32, U64, F32, SZ = (C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_float,
                                  C.c_size_t)


class StepIO(C.Structure):
    """hl_step_io of include/hotline.h, field for field."""
    _fields_ = [("rows", P), ("bag_ptr", P), ("n_samples", I32), ("bags_per_sample", I32), ("n_lookups", I64),
                ("dY", P), ("lr", F32), ("gids", P), ("codes", P), ("flags", P), ("pop_ids", P),
                ("nonpop_ids", P), ("counts", P), ("cold_ids", P), ("n_cold", P), ("w_host", P), ("w_hot", P),
                ("staging", P), ("staging_cap", I32), ("out", P), ("workspace", P), ("ws_bytes", SZ),
                ("write_back", I32), ("step_flags", U32)]


HL_STEP_UNTIED = 1
HL_STEP_PLANNED = 2
HL_STEP_HANDOVER_KERNELS = 4
_SIGS = {
    "hl_status_string": (C.c_char_p, [C.c_int]),
    "hl_create": (C.c_int, [C.POINTER(P), I32, P, I32, C.c_int, U32]),
    "hl_destroy": (C.c_int, [P]),
    "hl_n_rows": (U64, [P]),
    "hl_n_hot": (U32, [P]),
    "hl_k_cap": (U32, [P]),
    "hl_workspace_bytes": (SZ, [P, I64, I64, I32]),
    "hl_workspace_init": (C.c_int, [P, SZ, P]),
    "hl_lookup_gids": (C.c_int, [P, P, P, I64, P, P]),
    "hl_profile_count": (C.c_int, [P, P, I64, P]),
    "hl_profile_counts": (C.c_int, [P, P, P]),
    "hl_profile_topk": (C.c_int, [P, U32, P, C.POINTER(U32), C.c_int, P]),
    "hl_set_hot": (C.c_int, [P, P, U32, P]),
    "hl_hot_fill": (C.c_int, [P, P, P, P, P]),
    "hl_hot_migrate": (C.c_int, [P, P, U32, P, P, P, P, P]),
    "hl_eal_create": (C.c_int, [P, U32, I32, I64, C.POINTER(P)]),
    "hl_eal_destroy": (C.c_int, [P]),
    "hl_eal_reset": (C.c_int, [P, P]),
    "hl_eal_access": (C.c_int, [P, P, I64, P]),
    "hl_eal_hot": (C.c_int, [P, P, C.POINTER(U32), P]),
    "hl_eal_state": (C.c_int, [P, P, P, P]),
    "hl_classify": (C.c_int, [P, P, P, I32, I32, I64, P, P]),
    "hl_partition": (C.c_int, [P, P, I32, P, P, P, P, SZ, P]),
    "hl_remap": (C.c_int, [P, P, I64, P, P]),
    "hl_dispatch": (C.c_int, [P, P, P, I32, I32, I64, P, P, P, P, P, P, P, SZ, P]),
    "hl_cold_gather": (C.c_int, [P, P, P, P, I32, I32, I64, P, P, I32, P, P, I32, P, P, P, SZ, P]),
    "hl_cold_plan": (C.c_int, [P, P, P, P, I32, I32, I64, P, P, I32, I32, P, P, P, SZ, P]),
    "hl_cold_fetch": (C.c_int, [P, P, P, I32, P, P, P]),
    "hl_cold_reserve": (C.c_int, [P, I64, P]),
    "hl_cold_scatter": (C.c_int, [P, P, P, I32, P, P, P]),
    "hl_embbag_fwd": (C.c_int, [P, P, P, I32, P, P, I32, I32, I64, P, P, I32, P, P]),
    "hl_embbag_fwd_part": (C.c_int, [P, P, P, I32, P, P, I32, I32, I64, P, P, I32, P, I32, P]),
    "hl_embbag_bwd_sgd": (C.c_int, [P, P, P, I32, P, P, I32, I32, I64, P, P, I32, P, F32, P, SZ, P]),
    "hl_embbag_bwd_plan": (C.c_int, [P, I32, P, P, I32, I32, I64, P, P, I32, P, SZ, P]),
    "hl_embbag_fwd_plan": (C.c_int, [P, P, P, I32, P, P, I32, I32, I64, P, P, SZ, P]),
    "hl_embbag_bwd_apply": (C.c_int, [P, P, P, I32, I32, I32, I64, P, F32, P, SZ, P]),
    "hl_embbag_bwd_apply_part": (C.c_int, [P, P, P, I32, I32, I32, I64, P, F32, I32, P, SZ, P]),
    "hl_embbag_bwd_grouping": (C.c_int, [P, I32, I32, I32, I64, P, SZ, P, P, P]),
    "hl_noalloc_scratch_bytes": (SZ, []),
    "hl_embbag_bwd_sgd_noalloc": (C.c_int, [P, P, P, I32, P, P, I32, I32, I64, P, P, I32, P, F32, P]),
    "hl_last_device_error": (C.c_int, [P, C.POINTER(U32)]),
    "hl_debug_ballot_ranks": (C.c_int, [P, I32]),
    "hl_trace_enable": (C.c_int, [P, I32]),
    "hl_trace_count": (I32, [P]),
    "hl_trace_only": (C.c_int, [P, C.c_char_p]),
    "hl_trace_read": (C.c_int, [P, I32, C.POINTER(C.c_char_p), C.POINTER(C.c_float)]),
    "hl_trace_read_at": (C.c_int, [P, I32, C.POINTER(C.c_char_p), C.POINTER(C.c_float), C.POINTER(C.c_float)]),
    "hl_trace_reset": (C.c_int, [P]),
    "hl_host_alloc": (C.c_int, [SZ, C.POINTER(P), C.POINTER(P)]),
    "hl_stream_create": (C.c_int, [I32, I32, I32, C.POINTER(P)]),
    "hl_pipeline_create": (C.c_int, [P, I32, I32, C.POINTER(P)]),
    "hl_pipeline_destroy": (C.c_int, [P]),
    "hl_pipeline_step": (C.c_int, [P, C.POINTER(StepIO), P]),
    "hl_pipeline_plan": (C.c_int, [P, C.POINTER(StepIO), P]),
    "hl_pipeline_sync_writeback": (C.c_int, [P, P]),
    "hl_pipeline_sync": (C.c_int, [P, P]),
    "hl_pipeline_streams": (C.c_int, [P, C.POINTER(P), C.POINTER(P), C.POINTER(P)]),
    "hl_stream_destroy": (C.c_int, [P]),
    "hl_host_free": (C.c_int, [P]),
}


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run python -m paper_2204_05436_amd.build")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


# Library objects still alive when the interpreter exits are destroyed here,
# newest first, after the device has finished their work: the HIP runtime's
# own teardown (and a profiler's, which runs before it) must not find
# compute-unit-masked streams, events, pinned host memory or handles of this
# library still registered with it.
_live = {}
_seq = itertools.count()


def _track(key, destroy):
    _live[key] = (next(_seq), destroy)


def _untrack(key):
    _live.pop(key, None)


@atexit.register
def _destroy_live():
    if not _live:
        return
    torch = sys.modules.get("torch")
    try:
        if torch is not None and torch.cuda.is_initialized():
            torch.cuda.synchronize()
    except Exception:
        pass
    for key, (_, destroy) in sorted(_live.items(), key=lambda kv: -kv[1][0]):
        try:
            destroy()
        except Exception:
            pass
    _live.clear()


def _ck(fn, st):
    if st != 0:
        raise HotlineError(fn, st)


def _p(x):
    """Device/host pointer of a torch tensor, an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _s(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _nbytes(t):
    return t.numel() * t.element_size()


class Handle:
    def __init__(self, ptr):
        self.ptr = ptr
        _track(("handle", ptr), self.close)

    @property
    def n_rows(self):
        return int(lib().hl_n_rows(self.ptr))

    @property
    def n_hot(self):
        return int(lib().hl_n_hot(self.ptr))

    @property
    def k_cap(self):
        return int(lib().hl_k_cap(self.ptr))

    def close(self):
        if self.ptr:
            _untrack(("handle", self.ptr))
            _ck("hl_destroy", lib().hl_destroy(self.ptr))
            self.ptr = None


def hl_status_string(status):
    return lib().hl_status_string(status).decode()


def hl_create(rows_per_table, dim, dtype, k_cap):
    rows = np.ascontiguousarray(rows_per_table, dtype=np.uint32)
    h = P()
    dt = HL_F32 if dtype in ("f32", HL_F32) else HL_BF16
    _ck("hl_create", lib().hl_create(C.byref(h), len(rows), rows.ctypes.data, int(dim), dt, int(k_cap)))
    return Handle(h.value)


def hl_destroy(h):
    h.close()


def hl_n_rows(h):
    return h.n_rows


def hl_n_hot(h):
    return h.n_hot


def hl_k_cap(h):
    return h.k_cap


def hl_workspace_bytes(h, max_lookups, max_bags, max_samples):
    return int(lib().hl_workspace_bytes(h.ptr, int(max_lookups), int(max_bags), int(max_samples)))


def hl_workspace_init(ws, stream=None):
    _ck("hl_workspace_init", lib().hl_workspace_init(_p(ws), _nbytes(ws), _s(stream)))


def hl_lookup_gids(h, rows, bag_ptr, n_bags, gids, stream=None):
    _ck("hl_lookup_gids", lib().hl_lookup_gids(h.ptr, _p(rows), _p(bag_ptr), int(n_bags), _p(gids), _s(stream)))


def hl_profile_count(h, gids, n, stream=None):
    _ck("hl_profile_count", lib().hl_profile_count(h.ptr, _p(gids), int(n), _s(stream)))


def hl_profile_counts(h, counts_out, stream=None):
    _ck("hl_profile_counts", lib().hl_profile_counts(h.ptr, _p(counts_out), _s(stream)))


def hl_profile_topk(h, k, hot_ids_out, reset_counts=False, stream=None):
    nh = U32(0)
    _ck("hl_profile_topk", lib().hl_profile_topk(h.ptr, int(k), _p(hot_ids_out), C.byref(nh), int(bool(reset_counts)),
                                                 _s(stream)))
    return int(nh.value)


def hl_set_hot(h, hot_ids, n_hot, stream=None):
    _ck("hl_set_hot", lib().hl_set_hot(h.ptr, _p(hot_ids), int(n_hot), _s(stream)))


def hl_hot_fill(h, hot_ids, w_host_dev, w_hot, stream=None):
    _ck("hl_hot_fill", lib().hl_hot_fill(h.ptr, _p(hot_ids), _p(w_host_dev), _p(w_hot), _s(stream)))


def hl_hot_migrate(h, old_ids, n_old, new_ids, w_hot_old, w_hot_new, w_host_dev, stream=None):
    _ck("hl_hot_migrate", lib().hl_hot_migrate(h.ptr, _p(old_ids), int(n_old), _p(new_ids), _p(w_hot_old),
                                               _p(w_hot_new), _p(w_host_dev), _s(stream)))


class EAL:
    """An SRRIP access logger (hl_eal_*)."""

    def __init__(self, h, n_sets, ways, max_lookups):
        self.ptr = P()
        _ck("hl_eal_create", lib().hl_eal_create(h.ptr, int(n_sets), int(ways), int(max_lookups),
                                                 C.byref(self.ptr)))
        self.n_sets, self.ways = int(n_sets), int(ways)
        self._key = ("eal", self.ptr.value)
        _track(self._key, self.close)

    def close(self):
        if self.ptr:
            _untrack(self._key)
            _ck("hl_eal_destroy", lib().hl_eal_destroy(self.ptr))
            self.ptr = P()


def hl_eal_create(h, n_sets, ways, max_lookups):
    return EAL(h, n_sets, ways, max_lookups)


def hl_eal_destroy(e):
    e.close()


def hl_eal_reset(e, stream=None):
    _ck("hl_eal_reset", lib().hl_eal_reset(e.ptr, _s(stream)))


def hl_eal_access(e, gids, n, stream=None):
    _ck("hl_eal_access", lib().hl_eal_access(e.ptr, _p(gids), int(n), _s(stream)))


def hl_eal_hot(e, hot_ids_out, stream=None):
    n = U32()
    _ck("hl_eal_hot", lib().hl_eal_hot(e.ptr, _p(hot_ids_out), C.byref(n), _s(stream)))
    return int(n.value)


def hl_eal_state(e, tags_out, rrpv_out, stream=None):
    _ck("hl_eal_state", lib().hl_eal_state(e.ptr, _p(tags_out), _p(rrpv_out), _s(stream)))


def hl_classify(h, gids, bag_ptr, n_samples, bags_per_sample, n_lookups, flags, stream=None):
    _ck("hl_classify", lib().hl_classify(h.ptr, _p(gids), _p(bag_ptr), int(n_samples), int(bags_per_sample),
                                         int(n_lookups), _p(flags), _s(stream)))


def hl_partition(h, flags, n_samples, pop_ids, nonpop_ids, counts_dev, ws, stream=None):
    _ck("hl_partition", lib().hl_partition(h.ptr, _p(flags), int(n_samples), _p(pop_ids), _p(nonpop_ids),
                                           _p(counts_dev), _p(ws), 0 if ws is None else _nbytes(ws), _s(stream)))


def hl_remap(h, gids, n, codes, stream=None):
    _ck("hl_remap", lib().hl_remap(h.ptr, _p(gids), int(n), _p(codes), _s(stream)))


def hl_dispatch(h, rows, bag_ptr, n_samples, bags_per_sample, n_lookups, gids, codes, flags, pop_ids, nonpop_ids,
                counts_dev, ws, stream=None):
    _ck("hl_dispatch", lib().hl_dispatch(
        h.ptr, _p(rows), _p(bag_ptr), int(n_samples), int(bags_per_sample), int(n_lookups), _p(gids), _p(codes),
        _p(flags), _p(pop_ids), _p(nonpop_ids), _p(counts_dev), _p(ws), 0 if ws is None else _nbytes(ws),
        _s(stream)))


def hl_cold_gather(h, gids, codes, bag_ptr, n_samples, bags_per_sample, n_lookups, sample_ids, n_sel_dev, n_sel_max,
                   w_host_dev, staging, staging_cap_rows, cold_ids_out, n_cold_dev, ws, stream=None):
    _ck("hl_cold_gather", lib().hl_cold_gather(
        h.ptr, _p(gids), _p(codes), _p(bag_ptr), int(n_samples), int(bags_per_sample), int(n_lookups),
        _p(sample_ids), _p(n_sel_dev), int(n_sel_max), _p(w_host_dev), _p(staging), int(staging_cap_rows),
        _p(cold_ids_out), _p(n_cold_dev), _p(ws), _nbytes(ws), _s(stream)))


def hl_cold_plan(h, gids, codes, bag_ptr, n_samples, bags_per_sample, n_lookups, sample_ids, n_sel_dev, n_sel_max,
                 staging_cap_rows, cold_ids_out, n_cold_dev, ws, stream=None):
    _ck("hl_cold_plan", lib().hl_cold_plan(
        h.ptr, _p(gids), _p(codes), _p(bag_ptr), int(n_samples), int(bags_per_sample), int(n_lookups),
        _p(sample_ids), _p(n_sel_dev), int(n_sel_max), int(staging_cap_rows), _p(cold_ids_out), _p(n_cold_dev),
        _p(ws), _nbytes(ws), _s(stream)))


def hl_cold_reserve(h, max_lookups, stream=None):
    _ck("hl_cold_reserve", lib().hl_cold_reserve(h.ptr, int(max_lookups), _s(stream)))


def hl_cold_fetch(h, cold_ids, n_cold_dev, staging_cap_rows, w_host_dev, staging, stream=None):
    _ck("hl_cold_fetch", lib().hl_cold_fetch(h.ptr, _p(cold_ids), _p(n_cold_dev), int(staging_cap_rows),
                                             _p(w_host_dev), _p(staging), _s(stream)))


def hl_cold_scatter(h, cold_ids, n_cold_dev, staging_cap_rows, staging, w_host_dev, stream=None):
    _ck("hl_cold_scatter", lib().hl_cold_scatter(h.ptr, _p(cold_ids), _p(n_cold_dev), int(staging_cap_rows),
                                                 _p(staging), _p(w_host_dev), _s(stream)))


def hl_embbag_fwd(h, w_hot, staging, staging_rows, codes, bag_ptr, n_samples, bags_per_sample, n_lookups,
                  sample_ids, n_sel_dev, n_sel_max, out, stream=None):
    _ck("hl_embbag_fwd", lib().hl_embbag_fwd(
        h.ptr, _p(w_hot), _p(staging), int(staging_rows), _p(codes), _p(bag_ptr), int(n_samples),
        int(bags_per_sample), int(n_lookups), _p(sample_ids), _p(n_sel_dev), int(n_sel_max), _p(out), _s(stream)))


def hl_embbag_fwd_part(h, w_hot, staging, staging_rows, codes, bag_ptr, n_samples, bags_per_sample, n_lookups,
                       sample_ids, n_sel_dev, n_sel_max, out, part, stream=None):
    _ck("hl_embbag_fwd_part", lib().hl_embbag_fwd_part(
        h.ptr, _p(w_hot), _p(staging), int(staging_rows), _p(codes), _p(bag_ptr), int(n_samples),
        int(bags_per_sample), int(n_lookups), _p(sample_ids), _p(n_sel_dev), int(n_sel_max), _p(out), int(part),
        _s(stream)))


def hl_embbag_bwd_sgd(h, w_hot, staging, staging_rows, codes, bag_ptr, n_samples, bags_per_sample, n_lookups,
                      sample_ids, n_sel_dev, n_sel_max, dY, lr, ws, stream=None):
    _ck("hl_embbag_bwd_sgd", lib().hl_embbag_bwd_sgd(
        h.ptr, _p(w_hot), _p(staging), int(staging_rows), _p(codes), _p(bag_ptr), int(n_samples),
        int(bags_per_sample), int(n_lookups), _p(sample_ids), _p(n_sel_dev), int(n_sel_max), _p(dY), float(lr),
        _p(ws), _nbytes(ws), _s(stream)))


def hl_noalloc_scratch_bytes():
    return int(lib().hl_noalloc_scratch_bytes())


def hl_embbag_bwd_sgd_noalloc(h, w_hot, staging, staging_rows, codes, bag_ptr, n_samples, bags_per_sample, n_lookups,
                              sample_ids, n_sel_dev, n_sel_max, dY, lr, stream=None):
    _ck("hl_embbag_bwd_sgd_noalloc", lib().hl_embbag_bwd_sgd_noalloc(
        h.ptr, _p(w_hot), _p(staging), int(staging_rows), _p(codes), _p(bag_ptr), int(n_samples),
        int(bags_per_sample), int(n_lookups), _p(sample_ids), _p(n_sel_dev), int(n_sel_max), _p(dY), float(lr),
        _s(stream)))


def hl_embbag_bwd_plan(h, staging_rows, codes, bag_ptr, n_samples, bags_per_sample, n_lookups, sample_ids, n_sel_dev,
                       n_sel_max, ws, stream=None):
    _ck("hl_embbag_bwd_plan", lib().hl_embbag_bwd_plan(
        h.ptr, int(staging_rows), _p(codes), _p(bag_ptr), int(n_samples), int(bags_per_sample), int(n_lookups),
        _p(sample_ids), _p(n_sel_dev), int(n_sel_max), _p(ws), _nbytes(ws), _s(stream)))


def hl_embbag_fwd_plan(h, w_hot, staging, staging_rows, codes, bag_ptr, n_samples, bags_per_sample, n_lookups, out, ws,
                       stream=None):
    _ck("hl_embbag_fwd_plan", lib().hl_embbag_fwd_plan(
        h.ptr, _p(w_hot), _p(staging), int(staging_rows), _p(codes), _p(bag_ptr), int(n_samples),
        int(bags_per_sample), int(n_lookups), _p(out), _p(ws), _nbytes(ws), _s(stream)))


def hl_embbag_bwd_apply(h, w_hot, staging, staging_rows, n_samples, bags_per_sample, n_lookups, dY, lr, ws,
                        stream=None):
    _ck("hl_embbag_bwd_apply", lib().hl_embbag_bwd_apply(
        h.ptr, _p(w_hot), _p(staging), int(staging_rows), int(n_samples), int(bags_per_sample), int(n_lookups),
        _p(dY), float(lr), _p(ws), _nbytes(ws), _s(stream)))


def hl_embbag_bwd_apply_part(h, w_hot, staging, staging_rows, n_samples, bags_per_sample, n_lookups, dY, lr, part,
                             ws, stream=None):
    _ck("hl_embbag_bwd_apply_part", lib().hl_embbag_bwd_apply_part(
        h.ptr, _p(w_hot), _p(staging), int(staging_rows), int(n_samples), int(bags_per_sample), int(n_lookups),
        _p(dY), float(lr), int(part), _p(ws), _nbytes(ws), _s(stream)))


def hl_embbag_bwd_grouping(h, staging_rows, n_samples, bags_per_sample, n_lookups, ws, keys_out, bags_out,
                           stream=None):
    _ck("hl_embbag_bwd_grouping", lib().hl_embbag_bwd_grouping(
        h.ptr, int(staging_rows), int(n_samples), int(bags_per_sample), int(n_lookups), _p(ws), _nbytes(ws),
        _p(keys_out), _p(bags_out), _s(stream)))


def hl_debug_ballot_ranks(h, on):
    _ck("hl_debug_ballot_ranks", lib().hl_debug_ballot_ranks(h.ptr, int(bool(on))))


def hl_last_device_error(h):
    e = U32(0)
    st = lib().hl_last_device_error(h.ptr, C.byref(e))
    if st not in (0, 6):
        raise HotlineError("hl_last_device_error", st)
    return int(e.value)


def hl_trace_enable(h, cap):
    _ck("hl_trace_enable", lib().hl_trace_enable(h.ptr, int(cap)))


def hl_trace_only(h, name=None):
    _ck("hl_trace_only", lib().hl_trace_only(h.ptr, None if name is None else name.encode()))


def hl_trace_count(h):
    return int(lib().hl_trace_count(h.ptr))


def hl_trace_read(h, i):
    name, ms = C.c_char_p(), C.c_float()
    _ck("hl_trace_read", lib().hl_trace_read(h.ptr, int(i), C.byref(name), C.byref(ms)))
    return name.value.decode(), float(ms.value)


def hl_trace_read_at(h, i):
    """(name, start ms after record 0's start, duration ms) of record i"""
    name, t0, ms = C.c_char_p(), C.c_float(), C.c_float()
    _ck("hl_trace_read_at", lib().hl_trace_read_at(h.ptr, int(i), C.byref(name), C.byref(t0), C.byref(ms)))
    return name.value.decode(), float(t0.value), float(ms.value)


def hl_trace_reset(h):
    _ck("hl_trace_reset", lib().hl_trace_reset(h.ptr))


def hl_stream_create(first_cu, n_cu, complement=False):
    """Returns the raw stream handle (wrap it with torch.cuda.ExternalStream)."""
    s = P()
    _ck("hl_stream_create", lib().hl_stream_create(int(first_cu), int(n_cu), int(bool(complement)), C.byref(s)))
    _track(("stream", s.value), lambda v=s.value: lib().hl_stream_destroy(v))
    return s.value


def hl_stream_destroy(stream):
    _untrack(("stream", stream))
    _ck("hl_stream_destroy", lib().hl_stream_destroy(stream))


def hl_pipeline_create(h, fetch_cus, plan_cus=0):
    p = P()
    _ck("hl_pipeline_create", lib().hl_pipeline_create(h.ptr, int(fetch_cus), int(plan_cus), C.byref(p)))
    _track(("pipeline", p.value), lambda v=p.value: lib().hl_pipeline_destroy(v))
    return p.value


def hl_pipeline_destroy(p):
    _untrack(("pipeline", p))
    _ck("hl_pipeline_destroy", lib().hl_pipeline_destroy(p))


def hl_pipeline_step(p, io: StepIO, stream=None):
    _ck("hl_pipeline_step", lib().hl_pipeline_step(p, C.byref(io), _s(stream)))


def hl_pipeline_plan(p, io: StepIO, stream=None):
    _ck("hl_pipeline_plan", lib().hl_pipeline_plan(p, C.byref(io), _s(stream)))


def hl_pipeline_sync_writeback(p, stream=None):
    _ck("hl_pipeline_sync_writeback", lib().hl_pipeline_sync_writeback(p, _s(stream)))


def hl_pipeline_sync(p, stream=None):
    _ck("hl_pipeline_sync", lib().hl_pipeline_sync(p, _s(stream)))


def hl_pipeline_streams(p):
    m, f, g = P(), P(), P()
    _ck("hl_pipeline_streams", lib().hl_pipeline_streams(p, C.byref(m), C.byref(f), C.byref(g)))
    return m.value, f.value, g.value


def hl_host_alloc(nbytes):
    host, dev = P(), P()
    _ck("hl_host_alloc", lib().hl_host_alloc(int(nbytes), C.byref(host), C.byref(dev)))
    return host.value, dev.value


def hl_host_free(host):
    _ck("hl_host_free", lib().hl_host_free(host))


class HostTable:
    """The full embedding table in pinned, device-mapped host memory: `.array`
    is a numpy view for the host, `.dev` the address kernels read through."""

    def __init__(self, n_rows, dim, dtype):
        self.np_dtype = np.float32 if dtype == "f32" else np.uint16
        self.shape = (int(n_rows), int(dim))
        self.nbytes = self.shape[0] * self.shape[1] * np.dtype(self.np_dtype).itemsize
        self.host, self.dev = hl_host_alloc(self.nbytes)
        buf = (C.c_char * self.nbytes).from_address(self.host)
        self.array = np.frombuffer(buf, dtype=self.np_dtype).reshape(self.shape)
        _track(("host", self.host), self.close)

    def torch_view(self):
        import torch
        return torch.from_numpy(self.array.view(np.float32 if self.np_dtype == np.float32 else np.int16))

    def close(self):
        if self.host:
            _untrack(("host", self.host))
            self.array = None
            hl_host_free(self.host)
            self.host = None
