"""Pins of the CPU oracle to things other than itself (no GPU needed).

* a worked example done by hand from the paper's definitions (every value
  exactly representable, so every comparison is exact);
* brute force on tiny random inputs with independent Python mechanisms
  (collections.Counter, set membership, numpy.flatnonzero);
* the defining property of the top-K selection, checked exhaustively;
* library routines for the arithmetic: torch CPU ``embedding_bag`` (sum) in
  fp64 for the forward, and its autograd gradient followed by a plain SGD step
  for the backward;
* invariants: partition sizes, popular samples touch only hot rows, split
  equals unsplit (Eq. 5), linearity of the update, untouched rows unchanged.
"""
import collections
import json
import pathlib

import numpy as np
import pytest
import torch

import oracle as O


# ---------------------------------------------------------------------------- hand example
# Two tables with 4 and 3 rows (global ids 0..3 and 4..6), dim 2, three samples
# with one lookup per table.  Worked by hand:
#   sample 0 -> rows (1, 0) -> ids {1, 4};  sample 1 -> (1, 2) -> {1, 6};
#   sample 2 -> (3, 0) -> {3, 4}.
#   counts: id1 = 2, id4 = 2, id3 = 1, id6 = 1.
#   K = 2: hot = {1, 4} (slots 0, 1); only sample 0 is all-hot -> O = [0], X = [1, 2].
#   slots: s0 (0, 1), s1 (0, -1), s2 (-1, 1); cold ids of X in order of first
#   occurrence (s1's id 6, then s2's id 3) = [6, 3] -> codes 2, 3.
#   pooled (one row per bag): the rows themselves.
#   dY per bag (1,0) (0,1) (1,1) (2,0) (0,-1) (1,1), lr = 0.5:
#   G(id1) = (1,0)+(1,1) = (2,1) -> (3,4) - (1,0.5) = (2, 3.5)
#   G(id4) = (0,1)+(1,1) = (1,2) -> (-1,0) - (0.5,1) = (-1.5, -1)
#   G(id3) = (0,-1)              -> (7,8) - (0,-0.5) = (7, 8.5)
#   G(id6) = (2,0)               -> (2,2) - (1,0)    = (1, 2)
#   K = 1: the tie id1/id4 at count 2 goes to the smaller id -> hot = {1}; no
#   sample is all-hot; cold ids by first occurrence = [4, 6, 3].
GOLD = pathlib.Path(__file__).parent / "golden"


def _gold(name):
    return json.loads((GOLD / name).read_text())


HAND = _gold("hand_two_tables.json")
HAND_ROWS_PER_TABLE = np.array(HAND["rows_per_table"], np.uint32)
HAND_TABLE = np.array(HAND["table"], np.float32)
HAND_ROWS = np.array(HAND["rows"], np.uint32)
HAND_PTR = np.array(HAND["bag_ptr"], np.int32)
HAND_DY = np.array(HAND["dY"], np.float32)
HAND_B, HAND_BPS, HAND_LR = HAND["n_samples"], HAND["bags_per_sample"], HAND["lr"]


def _table(dtype):
    return HAND_TABLE.copy() if dtype == "f32" else np.array(
        [[O.round_bf16(v) for v in r] for r in HAND_TABLE.astype(np.float64)], np.uint16)


def _as_f64(a, dtype):
    if dtype == "f32":
        return a.astype(np.float64)
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_hand_example_k2(dtype):
    x = HAND["k2"]
    g, rc = O.gids(HAND_ROWS_PER_TABLE, HAND_ROWS, HAND_PTR)
    assert rc == 0 and g.tolist() == HAND["gids"]
    counts, _ = O.count(len(HAND_TABLE), [g])
    assert counts.tolist() == HAND["counts"]
    hot = O.topk(counts, len(x["hot"]))
    assert hot.tolist() == x["hot"]
    flags = O.classify(hot, g, HAND_PTR, HAND_B, HAND_BPS)
    assert flags.tolist() == x["flags"]
    pop, nonpop = O.partition(flags)
    assert pop.tolist() == x["pop"] and nonpop.tolist() == x["nonpop"]
    codes0 = O.remap(hot, g)
    assert codes0.tolist() == x["codes_remap"]
    cold, codes = O.cold_plan(g, codes0, HAND_PTR, nonpop, len(nonpop), HAND_BPS, len(hot))
    assert cold.tolist() == x["cold_ids"] and codes.tolist() == x["codes"]
    table = _table(dtype)
    w_hot, stg = O.gather(table, hot), O.gather(table, cold)
    assert _as_f64(stg, dtype).tolist() == x["staging"]
    out, _, rc = O.embbag_fwd(dtype, w_hot, len(hot), stg, codes, HAND_PTR, None, HAND_B, HAND_BPS, len(g))
    assert rc == 0
    assert out.tolist() == x["out"]
    uniq, scale, rc = O.embbag_bwd_sgd(dtype, w_hot, len(hot), stg, codes, HAND_PTR, None, HAND_B, HAND_BPS, HAND_DY,
                                       HAND_LR, want_scale=True)
    assert rc == 0 and uniq.tolist() == x["unique_codes"]
    assert _as_f64(w_hot, dtype).tolist() == x["w_hot_after"]
    assert _as_f64(stg, dtype).tolist() == x["staging_after"]
    # error scale |row| + lr * sum|dY| for code 0 (id 1): (3 + 0.5*2, 4 + 0.5*1)
    assert scale[0].tolist() == x["error_scale_code0"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_hand_example_writeback(dtype):
    """After the K=2 step, writing the updated cold rows back and taking the hot
    rows from the cache gives the whole table updated by one SGD step (hand
    values above); rows no lookup names keep their bits."""
    x = HAND["k2"]
    g, _ = O.gids(HAND_ROWS_PER_TABLE, HAND_ROWS, HAND_PTR)
    hot = np.array(x["hot"], np.uint32)
    _, nonpop = O.partition(O.classify(hot, g, HAND_PTR, HAND_B, HAND_BPS))
    cold, codes = O.cold_plan(g, O.remap(hot, g), HAND_PTR, nonpop, len(nonpop), HAND_BPS, len(hot))
    table = _table(dtype)
    w_hot, stg = O.gather(table, hot), O.gather(table, cold)
    O.embbag_bwd_sgd(dtype, w_hot, len(hot), stg, codes, HAND_PTR, None, HAND_B, HAND_BPS, HAND_DY, HAND_LR)
    host = table.copy()
    O.scatter(host, cold, stg)
    assert _as_f64(host[cold.astype(np.int64)], dtype).tolist() == x["staging_after"]
    named = set(hot.tolist()) | set(cold.tolist())
    for r in range(len(table)):
        if r not in named:
            assert (host[r] == table[r]).all()
    host[hot] = w_hot
    assert _as_f64(host, dtype).tolist() == x["table_after_writeback"]


def test_hand_example_k1_tie_and_multihot():
    x = HAND["k1"]
    g, _ = O.gids(HAND_ROWS_PER_TABLE, HAND_ROWS, HAND_PTR)
    counts, _ = O.count(len(HAND_TABLE), [g])
    hot = O.topk(counts, 1)
    assert hot.tolist() == x["hot"]
    flags = O.classify(hot, g, HAND_PTR, HAND_B, HAND_BPS)
    pop, nonpop = O.partition(flags)
    assert pop.tolist() == x["pop"] and nonpop.tolist() == x["nonpop"]
    cold, codes = O.cold_plan(g, O.remap(hot, g), HAND_PTR, nonpop, len(nonpop), HAND_BPS, len(hot))
    assert cold.tolist() == x["cold_ids"]
    assert codes.tolist() == x["codes"]
    # multi-hot bag {id1, id1, id2} pools to (3+3+5, 4+4+6)
    m = HAND["multi_hot_bag"]
    out = O.embbag_fwd_flat("f32", HAND_TABLE, np.array(m["ids"], np.uint32), np.array([0, len(m["ids"])], np.int32))
    assert out.tolist() == [m["out"]]


def test_out_of_range_row_is_reported():
    g, rc = O.gids(HAND_ROWS_PER_TABLE, np.array([4, 0], np.uint32), np.array([0, 1, 2], np.int32))
    assert rc == 2 and g[0] == 0xFFFFFFFF and g[1] == 4


# ---------------------------------------------------------------------------- bf16 rounding
def test_bf16_rounding_ties_and_library():
    assert O.round_bf16(1.0 + 2.0 ** -8) == 0x3F80          # tie -> even (down)
    assert O.round_bf16(1.0 + 3 * 2.0 ** -8) == 0x3F82      # tie -> even (up)
    assert O.round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -30) == 0x3F81  # just above the tie
    assert O.round_bf16(-0.0) == 0x8000 and O.round_bf16(0.0) == 0
    assert O.round_bf16(3.5e38) == 0x7F80                     # overflow -> inf
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([O.round_bf16(float(v)) for v in x], np.uint16)
    assert (got == ref).all()


# ---------------------------------------------------------------------------- random tiny cases
def tiny_case(seed, max_bag=4, dim=3):
    rng = np.random.default_rng(seed)
    T = int(rng.integers(1, 4))
    rpt = rng.integers(1, 8, T).astype(np.uint32)
    steps = int(rng.integers(1, 3))
    B = int(rng.integers(0, 9))
    bps = T * steps
    lens = rng.integers(0, max_bag + 1, B * bps)
    ptr = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    rows = np.empty(int(ptr[-1]), np.uint32)
    for j in range(B * bps):
        t = j % T
        rows[ptr[j]:ptr[j + 1]] = rng.integers(0, rpt[t], lens[j])
    n_rows = int(rpt.sum())
    table = rng.integers(-8, 9, (n_rows, dim)).astype(np.float32) / 4
    dY = rng.integers(-8, 9, (B * bps, dim)).astype(np.float32) / 2
    base = np.concatenate([[0], np.cumsum(rpt)[:-1]]).astype(np.int64)
    tab_of_lookup = np.repeat(np.arange(B * bps) % T, lens)
    gids_ref = (base[tab_of_lookup] + rows).astype(np.uint32)
    return dict(T=T, rpt=rpt, B=B, bps=bps, ptr=ptr, rows=rows, n_rows=n_rows, table=table, dY=dY,
                gids=gids_ref, rng=rng)


def topk_property(counts, k, hot):
    cand = {g for g in range(len(counts)) if counts[g] >= 1}
    H = set(hot.tolist())
    assert len(H) == len(hot) == min(k, len(cand))
    assert H <= cand
    assert hot.tolist() == sorted(H)
    for h in H:
        for x in cand - H:
            assert counts[h] > counts[x] or (counts[h] == counts[x] and h < x)


@pytest.mark.parametrize("seed", range(60))
def test_tiny_brute_force(seed):
    c = tiny_case(seed)
    g, rc = O.gids(c["rpt"], c["rows"], c["ptr"])
    assert rc == 0 and (g == c["gids"]).all()
    n_rows, B, bps, ptr = c["n_rows"], c["B"], c["bps"], c["ptr"]
    # counting: Counter over the same ids, twice (two profiling batches)
    counts, _ = O.count(n_rows, [g, g[::-1].copy()])
    ref = collections.Counter(g.tolist() * 2)
    assert counts.tolist() == [ref.get(i, 0) for i in range(n_rows)]
    assert int(counts.sum()) == 2 * len(g)
    for k in [0, 1, 2, 3, n_rows // 2, n_rows, n_rows + 5]:
        hot = O.topk(counts, k)
        topk_property(counts, k, hot)
        H = set(hot.tolist())
        flags = O.classify(hot, g, ptr, B, bps)
        for b in range(B):
            ids = g[ptr[b * bps]:ptr[(b + 1) * bps]].tolist()
            assert flags[b] == int(all(i in H for i in ids))
        pop, nonpop = O.partition(flags)
        assert pop.tolist() == np.flatnonzero(flags).tolist()
        assert nonpop.tolist() == np.flatnonzero(flags == 0).tolist()
        assert len(pop) + len(nonpop) == B
        codes0 = O.remap(hot, g)
        for i, gi in enumerate(g.tolist()):
            assert (codes0[i] == -1) == (gi not in H)
            if codes0[i] >= 0:
                assert hot[codes0[i]] == gi
        k_cap = max(k, 1)
        cold, codes = O.cold_plan(g, codes0, ptr, nonpop, len(nonpop), bps, k_cap)
        cold_ref = []
        for b in nonpop:                       # first occurrence, streaming the mu-batch
            for i in range(ptr[b * bps], ptr[(b + 1) * bps]):
                if g[i] not in H and g[i] not in cold_ref:
                    cold_ref.append(int(g[i]))
        assert cold.tolist() == cold_ref
        for i in range(len(g)):
            if codes[i] >= k_cap:
                assert cold[codes[i] - k_cap] == g[i]
            else:
                assert codes[i] == codes0[i] and codes[i] >= 0
        # popular samples touch only hot rows
        for b in pop:
            assert all(codes[i] < k_cap for i in range(ptr[b * bps], ptr[(b + 1) * bps]))


def _torch_fwd_bwd(table, gids, ptr, dY, lr):
    W = torch.tensor(table.astype(np.float64), requires_grad=True)
    out = torch.nn.functional.embedding_bag(torch.from_numpy(gids.astype(np.int64)), W,
                                            torch.from_numpy(ptr.astype(np.int64)), mode="sum",
                                            include_last_offset=True)
    (out * torch.from_numpy(dY.astype(np.float64))).sum().backward()
    opt = torch.optim.SGD([W], lr=lr)
    pooled = out.detach().numpy().copy()
    opt.step()
    return pooled, W.detach().numpy()


@pytest.mark.parametrize("seed", range(40))
def test_forward_backward_vs_torch(seed):
    c = tiny_case(seed, max_bag=6, dim=int(np.random.default_rng(seed).integers(1, 6)))
    dim = c["table"].shape[1]
    c["table"] = np.random.default_rng(seed + 1).standard_normal((c["n_rows"], dim)).astype(np.float32)
    c["dY"] = np.random.default_rng(seed + 2).standard_normal((c["B"] * c["bps"], dim)).astype(np.float32)
    g, ptr, B, bps = c["gids"], c["ptr"], c["B"], c["bps"]
    counts, _ = O.count(c["n_rows"], [g])
    hot = O.topk(counts, max(1, c["n_rows"] // 3))
    flags = O.classify(hot, g, ptr, B, bps)
    pop, nonpop = O.partition(flags)
    k_cap = len(hot) + 2
    cold, codes = O.cold_plan(g, O.remap(hot, g), ptr, nonpop, len(nonpop), bps, k_cap)
    w_hot, stg = O.gather(c["table"], hot), O.gather(c["table"], cold)
    out, scale, rc = O.embbag_fwd("f32", w_hot, k_cap, stg, codes, ptr, None, B, bps, B * bps,
                                  want_scale=True)
    assert rc == 0
    lr = 0.01
    # the update takes lr as fp32: the library reference gets the same value
    pooled, W_new = _torch_fwd_bwd(c["table"], g, ptr, c["dY"], float(np.float32(lr)))
    # one fp32 rounding of the exact-in-fp64 sum
    assert np.all(np.abs(out.astype(np.float64) - pooled) <= 2.0 ** -24 * np.abs(pooled) + 1e-12 * scale)
    # split == unsplit (Eq. 5): the flat-table pooling gives the same bits
    assert (O.embbag_fwd_flat("f32", c["table"], g, ptr) == out).all()
    uniq, sc, rc = O.embbag_bwd_sgd("f32", w_hot, k_cap, stg, codes, ptr, None, B, bps, c["dY"], lr,
                                    want_scale=True)
    assert rc == 0
    ids_of_code = {i: int(hot[i]) for i in range(len(hot))}
    ids_of_code.update({k_cap + u: int(cold[u]) for u in range(len(cold))})
    touched = set()
    for j, code in enumerate(uniq.tolist()):
        gid = ids_of_code[code]
        touched.add(gid)
        got = (w_hot[code] if code < k_cap else stg[code - k_cap]).astype(np.float64)
        ref = W_new[gid]
        assert np.all(np.abs(got - ref) <= 2.0 ** -24 * np.abs(ref) + 1e-12 * sc[j]), (gid, got, ref)
    # rows no lookup names are unchanged (bitwise)
    for s in range(len(hot)):
        if int(hot[s]) not in touched:
            assert (w_hot[s] == c["table"][hot[s]]).all()
    # split == unsplit for the update too
    flat = c["table"].copy()
    O.embbag_bwd_sgd_flat("f32", flat, g, ptr, c["dY"], lr)
    for code in uniq.tolist():
        gid = ids_of_code[code]
        got = w_hot[code] if code < k_cap else stg[code - k_cap]
        assert (got == flat[gid]).all()


@pytest.mark.parametrize("seed", range(6))
def test_writeback_round_trip_and_composition(seed):
    """The write-back against numpy fancy assignment; gather then write-back is the
    identity; hot cache + written-back staging == the flat-table update (Eq. 5),
    bit for bit."""
    c = tiny_case(seed + 300, max_bag=5, dim=3)
    g, ptr, B, bps, n = c["gids"], c["ptr"], c["B"], c["bps"], c["n_rows"]
    rng = np.random.default_rng(seed)
    tab = rng.standard_normal((n, 3)).astype(np.float32)
    ids = rng.permutation(n)[: max(1, n // 2)].astype(np.uint32)
    rows = rng.standard_normal((len(ids), 3)).astype(np.float32)
    a = tab.copy()
    O.scatter(a, ids, rows)
    b = tab.copy()
    b[ids.astype(np.int64)] = rows
    assert (a == b).all()
    a = tab.copy()
    O.scatter(a, ids, O.gather(tab, ids))
    assert (a == tab).all()
    counts, _ = O.count(n, [g])
    hot = O.topk(counts, max(1, n // 4))
    _, nonpop = O.partition(O.classify(hot, g, ptr, B, bps))
    k_cap = len(hot) + 1
    cold, codes = O.cold_plan(g, O.remap(hot, g), ptr, nonpop, len(nonpop), bps, k_cap)
    dY = rng.standard_normal((B * bps, 3)).astype(np.float32)
    w_hot, stg = O.gather(tab, hot), O.gather(tab, cold)
    O.embbag_bwd_sgd("f32", w_hot, k_cap, stg, codes, ptr, None, B, bps, dY, 0.1)
    host = tab.copy()
    O.scatter(host, cold, stg)
    host[hot.astype(np.int64)] = w_hot
    flat = tab.copy()
    O.embbag_bwd_sgd_flat("f32", flat, g, ptr, dY, 0.1)
    assert (host == flat).all()


@pytest.mark.parametrize("seed", range(10))
def test_update_linearity_and_sequential(seed):
    c = tiny_case(seed + 100, max_bag=5, dim=4)
    g, ptr, B, bps = c["gids"], c["ptr"], c["B"], c["bps"]
    n = c["n_rows"]
    hot = np.arange(n, dtype=np.uint32)                 # all rows hot: every code is a slot
    codes = O.remap(hot, g)
    tab = np.random.default_rng(seed).standard_normal((n, 4)).astype(np.float32)
    dY = np.random.default_rng(seed + 7).standard_normal((B * bps, 4)).astype(np.float32)
    a = tab.copy()
    O.embbag_bwd_sgd("f32", a, n, None, codes, ptr, None, B, bps, dY, 0.25)
    b = tab.copy()
    O.embbag_bwd_sgd("f32", b, n, None, codes, ptr, None, B, bps, 2 * dY, 0.125)
    assert (a == b).all()   # scaling by 2 is exact in binary floating point
    # coalesced update == one lookup at a time (within the error scale)
    s = tab.astype(np.float64)
    absg = np.zeros_like(s)
    for bag in range(B * bps):
        for i in range(ptr[bag], ptr[bag + 1]):
            s[g[i]] -= 0.25 * dY[bag]
            absg[g[i]] += np.abs(dY[bag])
    tol = 1e-6 * (np.abs(tab) + 0.25 * absg) + 1e-30
    assert np.all(np.abs(a - s) <= tol)


def test_invalid_code_reported():
    w = np.zeros((2, 2), np.float32)
    out, _, rc = O.embbag_fwd("f32", w, 2, None, np.array([-1], np.int32), np.array([0, 1], np.int32),
                              None, 1, 1, 1)
    assert rc == 3
    _, _, rc = O.embbag_bwd_sgd("f32", w, 2, None, np.array([5], np.int32), np.array([0, 1], np.int32),
                                None, 1, 1, np.zeros((1, 2), np.float32), 0.1)
    assert rc == -3


def test_empty_inputs():
    assert O.topk(np.zeros(5, np.uint32), 3).tolist() == []
    assert O.classify(np.zeros(0, np.uint32), np.zeros(0, np.uint32), np.zeros(3, np.int32), 2, 1).tolist() == [1, 1]
    pop, nonpop = O.partition(np.zeros(0, np.uint8))
    assert len(pop) == len(nonpop) == 0


# ---------------------------------------------------------------------------- re-learning (hot-set migration)
# Hand example: six rows of dim 2, row r of the host table holds (r, r); the old
# hot set {1, 3} was trained to (10, 10) and (30, 30) in slots 0 and 1; the new
# hot set is {3, 4}.  Row 1 leaves: the host gets (10, 10).  Row 3 stays: it
# moves to slot 0 with (30, 30), and its stale host copy (3, 3) is left alone.
# Row 4 enters from the host: (4, 4) in slot 1.  One row written back.
def test_migrate_hand_example():
    x = _gold("migrate_hand.json")
    host = np.repeat(np.arange(x["n_rows"], dtype=np.float32)[:, None], 2, axis=1).copy()
    w_new, n = O.migrate(x["old_ids"], np.array(x["w_old"], np.float32), x["new_ids"], host)
    assert n == x["written_back"]
    assert np.array_equal(w_new, np.array(x["w_new"], np.float32))
    assert np.array_equal(host, np.array(x["host_after"], np.float32))


def _logical(host, ids, w_hot):
    """The table as the path reads it: a hot row from the cache, any other from the host."""
    t = host.copy()
    t[np.asarray(ids, np.int64)] = w_hot[: len(ids)]
    return t


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
def test_migrate_keeps_the_logical_table(seed, dtype):
    """Re-learning moves rows between the cache and the host but changes no row
    of the table the path reads (bit for bit), keeps the trained values of the
    rows that stay, and writes back exactly the rows that leave."""
    rng = np.random.default_rng(seed)
    n_rows, dim = int(rng.integers(8, 300)), int(rng.integers(1, 5))
    host = rng.integers(0, 1 << 15, size=(n_rows, dim)).astype(dtype)
    old = np.sort(rng.choice(n_rows, size=int(rng.integers(0, n_rows // 2 + 1)), replace=False)).astype(np.uint32)
    new = np.sort(rng.choice(n_rows, size=int(rng.integers(0, n_rows // 2 + 1)), replace=False)).astype(np.uint32)
    w_old = rng.integers(1 << 15, 1 << 16, size=(len(old), dim)).astype(dtype)  # trained: unlike any host row
    before = _logical(host, old, w_old)
    host0 = host.copy()
    w_new, n = O.migrate(old, w_old, new, host)
    assert np.array_equal(_logical(host, new, w_new), before)
    leave, stay = set(old.tolist()) - set(new.tolist()), set(old.tolist()) & set(new.tolist())
    assert n == len(leave)
    slot_old = {int(g): s for s, g in enumerate(old)}
    for s, g in enumerate(new.tolist()):
        src = w_old[slot_old[g]] if g in stay else host0[g]
        assert np.array_equal(w_new[s], src)
    untouched = np.setdiff1d(np.arange(n_rows), np.fromiter(leave, dtype=np.int64, count=len(leave)))
    assert np.array_equal(host[untouched], host0[untouched])


def test_migrate_same_and_disjoint_sets():
    rng = np.random.default_rng(7)
    host = rng.standard_normal((50, 3)).astype(np.float32)
    ids = np.array([2, 9, 17, 40], np.uint32)
    w_old = rng.standard_normal((4, 3)).astype(np.float32) + 100
    h0 = host.copy()
    w_new, n = O.migrate(ids, w_old, ids, host)  # the same set: nothing moves
    assert n == 0 and np.array_equal(w_new, w_old) and np.array_equal(host, h0)
    other = np.array([0, 5, 41], np.uint32)       # disjoint: every old row leaves, every new one enters
    w_new, n = O.migrate(ids, w_old, other, host)
    assert n == 4 and np.array_equal(host[ids], w_old) and np.array_equal(w_new, h0[other])


# ---------------------------------------------------------------------------- SRRIP access logger
def _mix32_np(x):
    """MurmurHash3's 32-bit finalizer, written from its published definition with numpy."""
    x = np.asarray(x, np.uint64) & np.uint64(0xFFFFFFFF)
    x ^= x >> np.uint64(16)
    x = (x * np.uint64(0x85EBCA6B)) & np.uint64(0xFFFFFFFF)
    x ^= x >> np.uint64(13)
    x = (x * np.uint64(0xC2B2AE35)) & np.uint64(0xFFFFFFFF)
    x ^= x >> np.uint64(16)
    return x.astype(np.uint32)


def test_eal_hash():
    pub = _gold("srrip_hand.json")["mix32"]
    assert O.mix32(0) == pub["0"] and O.mix32(1) == pub["1"]  # published values of the finalizer
    xs = np.random.default_rng(3).integers(0, 1 << 32, size=2000, dtype=np.uint64)
    assert [O.mix32(int(v)) for v in xs] == _mix32_np(xs).tolist()


# Worked by hand, one set of two ways (empty ways: RRPV 3):
#   5: miss, way 0 (RRPV 3) -> [5:2, -:3];   7: miss, way 1 -> [5:2, 7:2]
#   5: hit -> [5:0, 7:2];   9: miss, no 3: age -> [5:1, 7:3], way 1 -> [5:1, 9:2]
#   7: miss, no 3: age -> [5:2, 9:3], way 1 -> [5:2, 7:2]
#   11: miss, no 3: age -> [5:3, 7:3], first 3 is way 0 -> [11:2, 7:3];  hot = [7, 11]
# Scan resistance, one set of four ways: A B C D fill it (RRPV 2), A B hit (0);
# a scan X1..X4 of ids seen once: X1 ages the set (A B at 1, C D at 3) and takes
# C, X2 takes D, X3 ages again (A B at 2, X1 X2 at 3) and takes X1, X4 takes X2:
# A and B stay (LRU would have evicted them).
def test_eal_hand_examples():
    x = _gold("srrip_hand.json")
    t = x["two_ways"]
    e = O.EAL(t["sets"], t["ways"])
    e.access(t["stream"])
    assert e.tag.tolist() == t["tag"] and e.rrpv.tolist() == t["rrpv"] and e.hot().tolist() == t["hot"]
    t = x["scan"]
    e = O.EAL(t["sets"], t["ways"])
    e.access(t["stream"])
    assert e.tag.tolist() == t["tag"] and e.rrpv.tolist() == t["rrpv"]
    e.access([0xFFFFFFFF] * t["then_invalid"])  # the id of a row out of range is not logged
    assert e.tag.tolist() == t["tag"] and e.rrpv.tolist() == t["rrpv"]


@pytest.mark.parametrize("seed", range(8))
def test_eal_invariants(seed):
    """Random Zipf-like streams: every held id sits in its own set, at most once;
    RRPVs are in 0..3 and empty ways hold 3; the last id accessed in each set is
    held (RRPV 0 or 2); with at least as many ways as distinct ids per set
    nothing is evicted, so the hot set is every id seen."""
    rng = np.random.default_rng(seed)
    n_sets, ways = int(rng.integers(1, 40)), int(rng.integers(1, 9))
    ids = (rng.zipf(1.3, size=int(rng.integers(1, 3000))) * 7919 % 100003).astype(np.uint32)
    e = O.EAL(n_sets, ways)
    for chunk in np.array_split(ids, 3):
        e.access(chunk)
    tag, rr = e.tag.reshape(n_sets, ways), e.rrpv.reshape(n_sets, ways)
    assert (rr <= 3).all()
    assert (rr[tag == 0xFFFFFFFF] == 3).all()
    for s in range(n_sets):
        held = tag[s][tag[s] != 0xFFFFFFFF]
        assert len(set(held.tolist())) == len(held)
        assert ((_mix32_np(held) % np.uint32(n_sets)) == s).all()
    sets = _mix32_np(ids) % np.uint32(n_sets)
    for s in np.unique(sets):
        last = ids[np.flatnonzero(sets == s)[-1]]
        w = np.flatnonzero(tag[s] == last)
        assert len(w) == 1 and rr[s, w[0]] in (0, 2)
    big = O.EAL(n_sets, max(len(np.unique(ids[sets == s])) for s in np.unique(sets)))
    big.access(ids)
    assert np.array_equal(big.hot(), np.unique(ids))
