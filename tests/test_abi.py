"""The C ABI on the host, without a GPU: the library loads, exports every entry
point include/hotline.h declares, and rejects bad arguments before touching the
device."""
import ctypes as C
import os
import re

import pytest

from paper_2204_05436_amd import hotline as hl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hotline.h")


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return sorted(set(re.findall(r"\b(hl_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_path():
    names = declared()
    for n in ["hl_create", "hl_profile_count", "hl_profile_topk", "hl_classify", "hl_partition", "hl_remap",
              "hl_cold_gather", "hl_cold_plan", "hl_cold_fetch", "hl_cold_scatter", "hl_embbag_fwd",
              "hl_embbag_bwd_sgd", "hl_embbag_bwd_plan", "hl_embbag_bwd_apply", "hl_dispatch", "hl_embbag_fwd_part",
              "hl_embbag_bwd_apply_part", "hl_cold_reserve", "hl_pipeline_step", "hl_pipeline_plan",
              "hl_stream_create", "hl_hot_migrate", "hl_eal_create", "hl_eal_access", "hl_eal_hot",
              "hl_last_device_error"]:
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = C.CDLL(hl.LIB_PATH)
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing
    # the binding wraps each one under the same name
    assert not [n for n in declared() if not hasattr(hl, n)]


def test_host_side_validation():
    L = hl.lib()
    h = C.c_void_p()
    rows = (C.c_uint32 * 2)(3, 4)
    assert L.hl_create(C.byref(h), 0, rows, 4, 0, 1) == 1          # no tables
    assert L.hl_create(C.byref(h), 2, None, 4, 0, 1) == 1          # no row counts
    assert L.hl_create(C.byref(h), 2, rows, 0, 0, 1) == 1          # dim 0
    assert L.hl_create(C.byref(h), 2, rows, 4, 7, 1) == 1          # bad dtype
    assert L.hl_create(C.byref(h), 2, rows, 4, 0, 0) == 1          # k_cap 0
    big = (C.c_uint32 * 2)(0xF0000000, 0x20000000)
    assert L.hl_create(C.byref(h), 2, big, 4, 0, 1) == 2           # total rows >= 2^32-1
    zero = (C.c_uint32 * 2)(3, 0)
    assert L.hl_create(C.byref(h), 2, zero, 4, 0, 1) == 1          # empty table
    assert L.hl_workspace_bytes(None, 10, 10, 10) == 0
    assert L.hl_classify(None, None, None, 1, 1, 1, None, None) == 1
    assert L.hl_embbag_fwd(None, None, None, 0, None, None, 1, 1, 1, None, None, 1, None, None) == 1
    assert L.hl_last_device_error(None, None) == 1
    assert L.hl_cold_fetch(None, None, None, 1, None, None, None) == 1
    assert L.hl_dispatch(None, None, None, 1, 1, 1, None, None, None, None, None, None, None, 0, None) == 1
    assert L.hl_cold_scatter(None, None, None, 1, None, None, None) == 1
    assert L.hl_cold_plan(None, None, None, None, 1, 1, 1, None, None, 1, 1, None, None, None, 0, None) == 1
    assert L.hl_embbag_bwd_plan(None, 0, None, None, 1, 1, 1, None, None, 1, None, 0, None) == 1
    assert L.hl_embbag_bwd_apply(None, None, None, 0, 1, 1, 1, None, 0.1, None, 0, None) == 1
    assert L.hl_pipeline_step(None, None, None) == 1
    assert L.hl_pipeline_plan(None, None, None) == 1
    assert L.hl_hot_migrate(None, None, 0, None, None, None, None, None) == 1
    e = C.c_void_p()
    assert L.hl_eal_create(None, 4, 2, 10, C.byref(e)) == 1
    assert L.hl_eal_access(None, None, 0, None) == 1
    assert L.hl_eal_hot(None, None, None, None) == 1
    assert hl.hl_status_string(3) == "capacity exceeded"
    assert hl.hl_status_string(99) == "unknown status"
    assert hl.hl_status_string(-5) == "unknown status"
    assert L.hl_create(C.byref(h), 2, rows, 4, -1, 1) == 1         # negative dtype


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(hl, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(hl, "_lib", None)
    with pytest.raises(ImportError):
        hl.lib()
