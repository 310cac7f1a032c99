"""GPU parity of the step the benchmark times, at full size: look-ahead steps
issued untied from a side stream, each planning the next batches (three sets
of per-step buffers, plans two steps ahead; the host-link copy and the plans
on compute units of their own), exactly as bench.py issues them, with one
difference: the test syncs after every step to read its results.  Each step
is compared with the oracle run from the GPU's pre-step state: flags, both
mu-batch lists, codes, cold ids (bit-exact), pooled outputs, updated hot and
staging rows (within tolerance; untouched hot rows bitwise unchanged), and
the backward's grouping: every key's (key, bag) pairs contiguous, in
ascending lookup order (the stable order of numpy's argsort of the keys),
hot keys first.  The kernel trace shows the fused plan and the cold forward
(from the sorted tail, or bag by bag for multi-hot bags) ran."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2204_05436_amd import configs, hotline as hl, workload as W
from paper_2204_05436_amd.runner import HotPath, to_device
from parity_lib import as_f64, check_close, check_grouping, log, make_table

pytestmark = pytest.mark.gpu

N_STEPS = 3


@pytest.mark.parametrize("name,k,hk,wb", [("dlrm-large", None, False, False), ("multi-hot", None, False, False),
                                          ("multi-hot", 2000, False, False), ("dlrm-large", None, True, False),
                                          ("dlrm-large", None, False, True)])
def test_timed_step_full_size(name, k, hk, wb):
    """k: the hot-set size (None: the workload's).  Multi-hot with the 2000
    most accessed rows hot leaves popular rows cold, so bags repeat cold rows:
    the grouping's order inside a key, which the cold forward's adjacency test
    reads, is then exercised.  hk: the handovers between the streams as
    kernels of their own (the schedule the benchmark times its kernels in).
    wb: the updated cold rows written back to the host table after each step
    (the next steps gather from the updated table)."""
    w = configs.WORKLOADS[name]
    rows = W.table_rows(w)
    n_rows = int(rows.sum(dtype=np.int64))
    k_cap = w.k_cap(n_rows)
    rtol = {"f32": 1e-5, "bf16": 1e-2}[w.dtype]
    prof = [W.make_batch(w, rows, i) for i in range(w.profile_batches)]
    idx = [w.profile_batches + s for s in range(N_STEPS + 2)]
    steps = [W.make_batch(w, rows, i) for i in idx]
    dYs = [W.make_dy(w, i, mb.n_bags) for i, mb in zip(idx, steps)]
    log(f"[timed-step] {name}: rows={n_rows} B={w.batch} L={steps[0].n_lookups} k_cap={k_cap}")
    table = make_table(w, n_rows)
    hp = HotPath(w, rows, table, max(b.n_lookups for b in prof + steps), w.batch, device="cuda", writeback=wb)
    try:
        assert hp.n_sets == 3 and hp.fetch_cus == 8 and hp.plan_cus == 64
        hp.learn([to_device(p, "cuda") for p in prof], k=k)
        n_hot = hp.n_hot
        counts = np.zeros(n_rows, np.uint32)
        for p in prof:
            O.count(n_rows, [O.gids(rows, p.rows, p.bag_ptr)[0]], counts)
        hot = O.topk(counts, k_cap if k is None else k)
        assert np.array_equal(hp.hot_ids[:n_hot].cpu().numpy().view(np.uint32), hot)
        dbs = [to_device(mb, "cuda", dY) for mb, dY in zip(steps, dYs)]
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        torch.cuda.synchronize()
        hl.hl_trace_enable(hp.h, 4096)
        dup_cold = 0
        for si in range(N_STEPS):
            mb, dY = steps[si], dYs[si]
            w_pre = hp.w_hot[:n_hot].cpu().numpy().copy()
            # the oracle's plan needs the hot set and the batch only
            B, bps, L = mb.n_samples, mb.bags_per_sample, mb.n_lookups
            g, _ = O.gids(rows, mb.rows, mb.bag_ptr)
            flags = O.classify(hot, g, mb.bag_ptr, B, bps)
            pop, nonpop = O.partition(flags)
            cold, codes = O.cold_plan(g, O.remap(hot, g), mb.bag_ptr, nonpop, len(nonpop), bps, k_cap)
            # the host table's cold rows before the step (after the last
            # write-back), and a sample of its other rows
            stg = O.gather(table.array, cold)
            if wb:
                samp = np.setdiff1d(np.random.default_rng(si).integers(0, n_rows, 100000), cold)
                samp_pre = table.array[samp].copy()
            log(f"[timed-step] {name}: step {si}")
            with torch.cuda.stream(side):
                # the benchmark's call: plans for the next n_sets - 1 batches
                hp.step(dbs[si], untied=True, next=[dbs[j] for j in range(si + 1, si + hp.n_sets)],
                        handover_kernels=hk)
                hp.sync()
            torch.cuda.synchronize()
            assert hp.device_error() == 0, f"step {si}"
            assert np.array_equal(hp.flags[:B].cpu().numpy(), flags), f"step {si} flags"
            cnt = hp.counts.cpu().numpy()
            assert cnt[0] == len(pop) and cnt[1] == len(nonpop), f"step {si} mu-batch sizes"
            assert np.array_equal(hp.pop[:cnt[0]].cpu().numpy(), pop), f"step {si} popular list"
            assert np.array_equal(hp.nonpop[:cnt[1]].cpu().numpy(), nonpop), f"step {si} non-popular list"
            assert np.array_equal(hp.codes[:L].cpu().numpy(), codes), f"step {si} codes"
            n_cold = int(hp.n_cold.item())
            assert np.array_equal(hp.cold_ids[:n_cold].cpu().numpy().view(np.uint32), cold), f"step {si} cold ids"
            out, sc, _ = O.embbag_fwd(w.dtype, w_pre, k_cap, stg, codes, mb.bag_ptr, None, B, bps, B * bps,
                                      want_scale=True)
            check_close(hp.out[:B * bps].cpu().numpy(), out, sc, 1e-5, f"step {si} pooled output")
            w_ref = w_pre.copy()
            stg_ref = np.ascontiguousarray(stg.copy())
            uniq, usc, rc = O.embbag_bwd_sgd(w.dtype, w_ref, k_cap, stg_ref, codes, mb.bag_ptr, None, B, bps, dY,
                                             w.lr, want_scale=True)
            assert rc == 0
            hu = uniq < k_cap
            gw = hp.w_hot[:n_hot].cpu().numpy()
            gst = hp.staging[:n_cold].cpu().numpy()
            check_close(as_f64(gw[uniq[hu]], w.dtype), as_f64(w_ref[uniq[hu]], w.dtype), usc[hu], rtol,
                        f"step {si} hot rows")
            ts = uniq[~hu] - k_cap
            check_close(as_f64(gst[ts], w.dtype), as_f64(stg_ref[ts], w.dtype), usc[~hu], rtol,
                        f"step {si} staging rows")
            if wb:  # the host table: the cold rows updated, the others as before
                tab = table.array
                assert np.array_equal(tab[cold].view(np.uint8), gst.view(np.uint8)), f"step {si} written back"
                assert np.array_equal(tab[samp].view(np.uint8), samp_pre.view(np.uint8)), f"step {si} other rows"
            untouched = np.setdiff1d(np.arange(n_hot), uniq[hu])
            assert np.array_equal(gw[untouched].view(np.uint8), w_pre[untouched].view(np.uint8)), f"step {si}"
            keys = torch.zeros(L, dtype=torch.int32, device="cuda")
            gbags = torch.zeros(L, dtype=torch.int32, device="cuda")
            hl.hl_embbag_bwd_grouping(hp.h, hp.staging_cap, B, bps, L, hp.ws, keys, gbags)
            torch.cuda.synchronize()
            bag_of = np.repeat(np.arange(B * bps, dtype=np.uint32), np.diff(mb.bag_ptr.astype(np.int64)))
            d_all, d_cold = check_grouping(keys.cpu().numpy().view(np.uint32), gbags.cpu().numpy().view(np.uint32),
                                           codes, bag_of, n_hot, k_cap, f"step {si} grouping")
            dup_cold += d_cold
            log(f"[timed-step] {name}: step {si} ok (popular {len(pop)}, cold rows {n_cold}, repeated pairs "
                f"{d_all}, of cold rows {d_cold})")
        names = [hl.hl_trace_read(hp.h, i)[0] for i in range(hl.hl_trace_count(hp.h))]
        hl.hl_trace_enable(hp.h, 0)
        # the fused plan (the cold insert in the dispatch kernel, the cold codes
        # in the grouping's first kernel) and the cold forward from the sorted tail
        assert names.count("cg_insert") == 0 and names.count("cg_codes") == 0, names
        # (multi-hot bags: the cold half bag by bag in the same launch)
        assert names.count("eb_tail_r2") + names.count("eb_bags_r2") == N_STEPS, names
        assert names.count("eb_bags_r2") == (N_STEPS if mb.n_lookups > 2 * mb.n_bags else 0), names
        assert names.count("eb_fwd_hot") == N_STEPS, names
        if k is not None:
            assert dup_cold > 0, "no bag repeats a cold row: the adjacency case is not exercised"
    finally:
        hp.close()
        table.close()
