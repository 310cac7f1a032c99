"""Shared helpers of the GPU parity tests: run every stage of the hot path on
the GPU through the C ABI (snapshotting each result) and through the oracle
on the same seeded inputs, then compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle as O
from paper_2204_05436_amd import hotline as hl
from paper_2204_05436_amd import workload as W
from paper_2204_05436_amd.runner import HotPath, to_device

RTOL = {"f32": 1e-5, "bf16": 1e-2}


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def make_table(w, n_rows, device="cuda"):
    t = hl.HostTable(n_rows, w.dim, w.dtype)
    if n_rows * w.dim <= 20_000_000:
        W.fill_weights_np(w, t.array)
    else:
        W.fill_weights_torch(w, t.torch_view(), device)
        torch.cuda.synchronize()
    return t


def u32(t):
    return t.cpu().numpy().view(np.uint32)


def as_f64(a, dtype):
    a = np.asarray(a)
    if dtype == "f32":
        return a.astype(np.float64)
    return (a.view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def check_close(got, ref, scale, rtol, what):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    tol = rtol * np.maximum(np.abs(ref), scale)
    bad = np.abs(got - ref) > tol
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} elements out of tolerance, first at {tuple(i)}: "
                             f"got {got[tuple(i)]!r} ref {ref[tuple(i)]!r} tol {tol[tuple(i)]!r}")


def check_grouping(keys, bags, codes, bag_of, n_hot, k_cap, what):
    """The backward's grouping of one mini-batch (hl_embbag_bwd_grouping)
    against the lookups' codes: the pairs of a key contiguous, its bags in
    ascending lookup order (the stable order of numpy's argsort of the keys),
    hot keys before the others.  Returns the number of repeated (key, bag)
    pairs (a row twice in one bag) and how many of them are of staging rows."""
    c = np.asarray(codes).astype(np.int64)
    want_k = np.where((c >= 0) & (c < n_hot), c, np.where(c >= k_cap, n_hot + (c - k_cap), 0xFFFFFFFF))
    want_k = want_k.astype(np.uint32)
    order = np.argsort(want_k, kind="stable")
    got_order = np.argsort(keys, kind="stable")
    assert np.array_equal(keys[got_order], want_k[order]), f"{what}: keys differ as multisets"
    assert np.array_equal(bags[got_order], bag_of[order]), f"{what}: a key's bags are not in lookup order"
    runs = 1 + int(np.count_nonzero(keys[1:] != keys[:-1])) if keys.size else 0
    assert runs == np.unique(keys).size, f"{what}: a key's pairs are not contiguous"
    hot = keys < n_hot
    assert not (hot[1:] & ~hot[:-1]).any(), f"{what}: a hot key after a non-hot one"
    dup = (keys[1:] == keys[:-1]) & (bags[1:] == bags[:-1])
    return int(dup.sum()), int((dup & ~hot[1:]).sum())


def grouping_of(hp, B, bps, L):
    """The grouping the last backward plan left in hp's workspace, as numpy."""
    keys = torch.zeros(max(1, L), dtype=torch.int32, device=hp.device)
    bags = torch.zeros(max(1, L), dtype=torch.int32, device=hp.device)
    hl.hl_embbag_bwd_grouping(hp.h, hp.staging_cap, B, bps, L, hp.ws, keys, bags)
    return keys[:L].cpu().numpy().view(np.uint32).copy(), bags[:L].cpu().numpy().view(np.uint32).copy()


def _on_side(fn):
    """Run fn(stream) on a fresh side stream ordered after the current stream's
    work; the current stream then waits for it."""
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    e0, e1 = torch.cuda.Event(), torch.cuda.Event()
    e0.record(main)
    side.wait_event(e0)
    fn(side)
    e1.record(side)
    main.wait_event(e1)


def run_gpu_stages(hp: HotPath, prof, mb, dY, k=None, hot_ids=None, split=False, fwd_plan=False):
    """All stages on the GPU, with snapshots.  Either profiles (k) or installs hot_ids.
    split: the dispatch kernel for ids, classify, partition and remap, the cold
    gather as plan + fetch and the backward as plan + apply, the fetch and the
    backward's plan each on a side stream (the pipelined schedule's entry
    points).  fwd_plan (not split): the forward over every sample with the
    backward's plan (hl_embbag_fwd_plan), then the apply."""
    h = hp.h
    r = {}
    dprof = [to_device(p, hp.device) for p in prof]
    if hot_ids is None:
        for b in dprof:
            hl.hl_lookup_gids(h, b.rows, b.bag_ptr, b.n_bags, hp.gids)
            hl.hl_profile_count(h, hp.gids, b.n_lookups)
        cnt = torch.zeros(h.n_rows, dtype=torch.int32, device=hp.device)
        hl.hl_profile_counts(h, cnt)
        r["counts"] = u32(cnt)
        hp.n_hot = hl.hl_profile_topk(h, hp.k_cap if k is None else k, hp.hot_ids, reset_counts=True)
        hl.hl_hot_fill(h, hp.hot_ids, hp.table.dev, hp.w_hot)
    else:
        hp.set_hot(torch.from_numpy(np.asarray(hot_ids, np.uint32).view(np.int32)).to(hp.device))
    n_hot = hp.n_hot
    r["hot"] = u32(hp.hot_ids[:n_hot])
    r["w_hot_pre"] = hp.w_hot[:n_hot].cpu().numpy().copy()
    b = to_device(mb, hp.device, dY)
    B, bps, L = b.n_samples, b.bps, b.n_lookups
    r["bag_ptr"] = np.asarray(mb.bag_ptr)
    if split:  # the dispatch kernel, as the pipelined step calls it
        hl.hl_dispatch(h, b.rows, b.bag_ptr, B, bps, L, hp.gids, hp.codes, hp.flags, hp.pop, hp.nonpop, hp.counts,
                       hp.ws)
        r["gids"] = u32(hp.gids[:L])
        r["flags"] = hp.flags[:B].cpu().numpy().copy()
    else:
        hl.hl_lookup_gids(h, b.rows, b.bag_ptr, b.n_bags, hp.gids)
        r["gids"] = u32(hp.gids[:L])
        hl.hl_classify(h, hp.gids, b.bag_ptr, B, bps, L, hp.flags)
        r["flags"] = hp.flags[:B].cpu().numpy().copy()
        hl.hl_partition(h, hp.flags, B, hp.pop, hp.nonpop, hp.counts, hp.ws)
    cnts = hp.counts.cpu().numpy()
    r["n_pop"], r["n_nonpop"] = int(cnts[0]), int(cnts[1])
    r["pop"] = hp.pop[:r["n_pop"]].cpu().numpy().copy()
    r["nonpop"] = hp.nonpop[:r["n_nonpop"]].cpu().numpy().copy()
    if not split:
        hl.hl_remap(h, hp.gids, L, hp.codes)
    r["codes_remap"] = hp.codes[:L].cpu().numpy().copy()
    if split:
        # as the pipelined step calls it: no sample list (cold lookups occur only
        # in non-popular samples)
        hl.hl_cold_plan(h, hp.gids, hp.codes, b.bag_ptr, B, bps, L, None, None, B, hp.staging_cap,
                        hp.cold_ids, hp.n_cold, hp.ws)
        _on_side(lambda st: hl.hl_cold_fetch(h, hp.cold_ids, hp.n_cold, hp.staging_cap, hp.table.dev, hp.staging,
                                             stream=st))
    else:
        hl.hl_cold_gather(h, hp.gids, hp.codes, b.bag_ptr, B, bps, L, hp.nonpop, hp.counts[1:], B, hp.table.dev,
                          hp.staging, hp.staging_cap, hp.cold_ids, hp.n_cold, hp.ws)
    n_cold = int(hp.n_cold.cpu().item())
    r["n_cold"] = n_cold
    r["cold"] = u32(hp.cold_ids[:min(n_cold, hp.staging_cap)])
    r["codes"] = hp.codes[:L].cpu().numpy().copy()
    r["staging_pre"] = hp.staging[:min(n_cold, hp.staging_cap)].cpu().numpy().copy()
    hp.out.zero_()
    if split:
        # as the pipelined step: popular forward, hot half of the non-popular one, the
        # backward's plan and first half on side streams, then the staging rows
        hl.hl_embbag_fwd_part(h, hp.w_hot, hp.staging, hp.staging_cap, hp.codes, b.bag_ptr, B, bps, L, hp.pop,
                              hp.counts[0:], B, hp.out, 0)
        hl.hl_embbag_fwd_part(h, hp.w_hot, hp.staging, hp.staging_cap, hp.codes, b.bag_ptr, B, bps, L, hp.nonpop,
                              hp.counts[1:], B, hp.out, 1)
        _on_side(lambda st: hl.hl_embbag_bwd_plan(h, hp.staging_cap, hp.codes, b.bag_ptr, B, bps, L, None, None, B,
                                                  hp.ws, stream=st))
        _on_side(lambda st: hl.hl_embbag_bwd_apply_part(h, hp.w_hot, hp.staging, hp.staging_cap, B, bps, L, b.dY,
                                                        hp.w.lr, 1, hp.ws, stream=st))
        hl.hl_embbag_fwd_part(h, hp.w_hot, hp.staging, hp.staging_cap, hp.codes, b.bag_ptr, B, bps, L, hp.nonpop,
                              hp.counts[1:], B, hp.out, 2)
        r["out"] = hp.out[:B * bps].cpu().numpy().copy()
        hl.hl_embbag_bwd_apply_part(h, hp.w_hot, hp.staging, hp.staging_cap, B, bps, L, b.dY, hp.w.lr, 2, hp.ws)
    elif fwd_plan:
        hl.hl_embbag_fwd_plan(h, hp.w_hot, hp.staging, hp.staging_cap, hp.codes, b.bag_ptr, B, bps, L, hp.out, hp.ws)
        r["out"] = hp.out[:B * bps].cpu().numpy().copy()
        hl.hl_embbag_bwd_apply(h, hp.w_hot, hp.staging, hp.staging_cap, B, bps, L, b.dY, hp.w.lr, hp.ws)
    else:
        hl.hl_embbag_fwd(h, hp.w_hot, hp.staging, hp.staging_cap, hp.codes, b.bag_ptr, B, bps, L, hp.pop,
                         hp.counts[0:], B, hp.out)
        hl.hl_embbag_fwd(h, hp.w_hot, hp.staging, hp.staging_cap, hp.codes, b.bag_ptr, B, bps, L, hp.nonpop,
                         hp.counts[1:], B, hp.out)
        r["out"] = hp.out[:B * bps].cpu().numpy().copy()
        hl.hl_embbag_bwd_sgd(h, hp.w_hot, hp.staging, hp.staging_cap, hp.codes, b.bag_ptr, B, bps, L, None, None,
                             B, b.dY, hp.w.lr, hp.ws)
    r["w_hot_new"] = hp.w_hot[:n_hot].cpu().numpy().copy()
    r["staging_new"] = hp.staging[:min(n_cold, hp.staging_cap)].cpu().numpy().copy()
    r["grouping"] = grouping_of(hp, B, bps, L) if b.dY is not None else None
    r["n_hot"] = n_hot
    r["deverr"] = hp.device_error()
    return r


def run_oracle(w, rows, prof, mb, dY, table_array, k_cap, k=None, hot_ids=None):
    n_rows = int(np.sum(rows, dtype=np.int64))
    r = {}
    if hot_ids is None:
        counts = np.zeros(n_rows, dtype=np.uint32)
        for p in prof:
            g, _ = O.gids(rows, p.rows, p.bag_ptr)
            O.count(n_rows, [g], counts)
        r["counts"] = counts
        hot = O.topk(counts, k_cap if k is None else k)
    else:
        hot = np.asarray(hot_ids, np.uint32)
    r["hot"] = hot
    g, _ = O.gids(rows, mb.rows, mb.bag_ptr)
    r["gids"] = g
    B, bps = mb.n_samples, mb.bags_per_sample
    r["flags"] = O.classify(hot, g, mb.bag_ptr, B, bps)
    r["pop"], r["nonpop"] = O.partition(r["flags"])
    r["codes_remap"] = O.remap(hot, g)
    r["cold"], r["codes"] = O.cold_plan(g, r["codes_remap"], mb.bag_ptr, r["nonpop"], len(r["nonpop"]), bps, k_cap)
    w_hot = O.gather(table_array, hot)
    stg = O.gather(table_array, r["cold"])
    r["w_hot_pre"], r["staging_pre"] = w_hot.copy(), stg.copy()
    out, scale, rc = O.embbag_fwd(w.dtype, w_hot, k_cap, stg, r["codes"], mb.bag_ptr, None, B, bps, B * bps,
                                  want_scale=True)
    assert rc == 0
    r["out"], r["out_scale"] = out, scale
    uniq, uscale, rc = O.embbag_bwd_sgd(w.dtype, w_hot, k_cap, stg, r["codes"], mb.bag_ptr, None, B, bps, dY, w.lr,
                                        want_scale=True)
    assert rc == 0
    r["w_hot_new"], r["staging_new"], r["uniq"], r["uscale"] = w_hot, stg, uniq, uscale
    return r


def compare(w, g, o, k_cap, check_counts=True):
    """Bit-exact for integer results, tolerance for floating point."""
    if check_counts and "counts" in o:
        assert np.array_equal(g["counts"], o["counts"]), "counts differ"
    assert np.array_equal(g["hot"], o["hot"]), f"hot set differs ({len(g['hot'])} vs {len(o['hot'])})"
    assert np.array_equal(g["gids"], o["gids"]), "gids differ"
    assert np.array_equal(g["flags"], o["flags"]), "flags differ"
    assert np.array_equal(g["pop"], o["pop"]) and np.array_equal(g["nonpop"], o["nonpop"]), "partition differs"
    assert g["n_pop"] + g["n_nonpop"] == len(g["flags"])
    assert np.array_equal(g["codes_remap"], o["codes_remap"]), "remap differs"
    assert g["n_cold"] == len(o["cold"]) and np.array_equal(g["cold"], o["cold"]), "cold ids differ"
    assert np.array_equal(g["codes"], o["codes"]), "cold codes differ"
    assert np.array_equal(g["w_hot_pre"].view(np.uint8), o["w_hot_pre"].view(np.uint8)), "hot cache fill differs"
    assert np.array_equal(g["staging_pre"].view(np.uint8), o["staging_pre"].view(np.uint8)), "gathered rows differ"
    # pooled outputs: fp32 accumulation of exact (widened) rows
    check_close(g["out"], o["out"], o["out_scale"], 1e-5, "pooled output")
    rtol = RTOL[w.dtype]
    n_hot = len(o["hot"])
    touched_hot = o["uniq"][o["uniq"] < k_cap]
    touched_stg = o["uniq"][o["uniq"] >= k_cap] - k_cap
    sc_hot = o["uscale"][o["uniq"] < k_cap]
    sc_stg = o["uscale"][o["uniq"] >= k_cap]
    check_close(as_f64(g["w_hot_new"][touched_hot], w.dtype), as_f64(o["w_hot_new"][touched_hot], w.dtype), sc_hot,
                rtol, "updated hot rows")
    check_close(as_f64(g["staging_new"][touched_stg], w.dtype), as_f64(o["staging_new"][touched_stg], w.dtype),
                sc_stg, rtol, "updated staging rows")
    untouched = np.setdiff1d(np.arange(n_hot), touched_hot)
    assert np.array_equal(g["w_hot_new"][untouched].view(np.uint8), g["w_hot_pre"][untouched].view(np.uint8)), \
        "untouched hot rows changed"
    assert g["deverr"] == 0, f"device error word {g['deverr']:#x}"
    if g.get("grouping") is not None:
        ptr = np.asarray(g["bag_ptr"], np.int64)
        bag_of = np.repeat(np.arange(len(ptr) - 1, dtype=np.uint32), np.diff(ptr))
        check_grouping(*g["grouping"], g["codes"], bag_of, g["n_hot"], k_cap, "grouping")
