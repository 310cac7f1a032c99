"""Orchestration of the hot path on one GPU: device buffers for a workload and
the library calls in the order the paper's pipeline runs them (Sec. IV: the
learning phase, then per mini-batch classification, fragmentation into the
popular and non-popular mu-batches, working-parameter gather for the
non-popular one, forward of both, and the update).  No arithmetic here: every
step is a call into libhotline.

The pipelined schedule (the paper's pipeline figure: the popular mu-batch runs
while the non-popular one's working parameters are gathered) uses three
streams of default priority:
  main  : dispatch (ids, classify, partition, remap), cold plan | fwd(popular),
          hot half of fwd(non-popular) | wait fetch, cold half of
          fwd(non-popular) | wait group, staging-row updates
  fetch : wait cold plan, row fetch over the host link [, write-back after
          the updates]
  group : wait cold plan, the backward's grouping of lookups by code | wait
          the hot halves of the forwards, reduction of dY and hot-row updates
          (the staging rows' sums are kept for the main stream)
Only the cold half of the non-popular forward and the staging-row updates
wait for the host link.
The cold id list and count are double-buffered so that a step's write-back
can still read them while the next step plans."""
from __future__ import annotations

from dataclasses import dataclass

from types import SimpleNamespace

import numpy as np
import torch

from . import hotline as hl
from .configs import Workload


@dataclass
class DevBatch:
    rows: torch.Tensor      # int32 view of uint32 table-local rows [L]
    bag_ptr: torch.Tensor   # int32 [n_bags+1]
    n_lookups: int
    n_samples: int
    bps: int
    dY: torch.Tensor | None = None  # float32 [n_bags, dim]

    @property
    def n_bags(self):
        return self.n_samples * self.bps


def to_device(batch, device, dY=None) -> DevBatch:
    rows = torch.from_numpy(batch.rows.view(np.int32)).to(device)
    ptr = torch.from_numpy(batch.bag_ptr.astype(np.int32)).to(device)
    d = None if dY is None else torch.from_numpy(np.ascontiguousarray(dY, dtype=np.float32)).to(device)
    return DevBatch(rows, ptr, batch.n_lookups, batch.n_samples, batch.bags_per_sample, d)


STAGES = ("gids", "classify", "partition", "remap", "cold_gather", "fwd_pop", "fwd_nonpop", "bwd")
MODES = ("pipelined", "sequential", "fwdbwd")


class HotPath:
    def __init__(self, w: Workload, rows_per_table, table: hl.HostTable, max_lookups: int, max_samples: int,
                 device="cuda", k_cap: int | None = None, staging_cap: int | None = None, writeback: bool = False,
                 fetch_cus: int = 8, plan_cus: int = 64, n_sets: int = 3):
        self.w = w
        self.device = device
        self.rows_per_table = np.asarray(rows_per_table, dtype=np.uint32)
        n_rows = int(self.rows_per_table.sum(dtype=np.int64))
        self.k_cap = int(k_cap if k_cap is not None else w.k_cap(n_rows))
        self.table = table
        self.h = hl.hl_create(self.rows_per_table, w.dim, w.dtype, self.k_cap)
        self.max_lookups = int(max_lookups)
        self.max_samples = int(max_samples)
        max_bags = self.max_samples * w.bags_per_sample
        wsb = hl.hl_workspace_bytes(self.h, self.max_lookups, max_bags, self.max_samples)
        sdt = torch.float32 if w.dtype == "f32" else torch.int16
        self.sdt = sdt
        self.w_hot = torch.zeros((self.k_cap, w.dim), dtype=sdt, device=device)
        self.staging_cap = int(staging_cap if staging_cap is not None else max(1, self.max_lookups))
        self.hot_ids = torch.zeros(max(1, min(self.k_cap, n_rows)), dtype=torch.int32, device=device)
        L, B = max(1, self.max_lookups), max(1, self.max_samples)
        i32 = dict(dtype=torch.int32, device=device)

        def bufs():
            return SimpleNamespace(
                gids=torch.zeros(L, **i32), codes=torch.zeros(L, **i32),
                flags=torch.zeros(B, dtype=torch.uint8, device=device), pop=torch.zeros(B, **i32),
                nonpop=torch.zeros(B, **i32), counts=torch.zeros(2, **i32),
                cold_ids=torch.zeros(self.staging_cap, **i32), n_cold=torch.zeros(1, **i32),
                staging=torch.zeros((self.staging_cap, w.dim), dtype=sdt, device=device),
                ws=torch.zeros(wsb, dtype=torch.uint8, device=device))

        # n_sets >= 2 sets of per-step buffers, taken in turn by the steps: a
        # write-back still reading one step's cold list, the look-ahead plans of
        # the next n_sets - 1 mini-batches, or the next step's row fetch, use the
        # others
        if n_sets < 2:
            raise ValueError("at least two sets of per-step buffers")
        self.n_sets = int(n_sets)
        self._sets = [bufs() for _ in range(self.n_sets)]
        self._par = 0
        self._use(0)
        self._pending = []  # look-ahead plans: (batch, set)
        self.writeback = bool(writeback)
        hl.hl_cold_reserve(self.h, self.max_lookups)  # no allocation inside a captured step
        # the native pipeline (its own streams; the host-link copy on compute units
        # of its own, since its slow host reads would stall kernels sharing them)
        self.fetch_cus = int(fetch_cus)
        self.plan_cus = int(plan_cus) if self.fetch_cus else 0
        self.pipe = hl.hl_pipeline_create(self.h, self.fetch_cus, self.plan_cus)
        self.io = hl.StepIO()
        # a process has a few hardware queues (streams beyond them share queues):
        # the Python rendering's streams are created only when it is used
        self._py_streams = None
        ev = lambda: torch.cuda.Event()
        self.ev_plan, self.ev_fetch, self.ev_group, self.ev_apply = ev(), ev(), ev(), ev()
        self.ev_fwdhot = ev()
        self.ev_wb = [ev() for _ in range(self.n_sets)]
        self.out = torch.zeros((max(1, max_bags), w.dim), dtype=torch.float32, device=device)
        self.n_hot = 0

    def _use(self, p):
        """The public per-step buffers (gids, codes, ..., ws) are set p's."""
        for k, v in vars(self._sets[p]).items():
            setattr(self, k, v)

    def _next_set(self):
        if self._pending:
            raise RuntimeError("a look-ahead plan is pending: step that batch first")
        p = self._par
        self._par = (p + 1) % self.n_sets
        self._use(p)
        return p

    def _fill_io(self, io, b, s, lr, flags):
        io.rows, io.bag_ptr, io.n_samples, io.bags_per_sample, io.n_lookups = (
            b.rows.data_ptr(), b.bag_ptr.data_ptr(), b.n_samples, b.bps, b.n_lookups)
        io.dY, io.lr = (b.dY.data_ptr() if b.dY is not None else None), float(lr)
        io.gids, io.codes, io.flags = s.gids.data_ptr(), s.codes.data_ptr(), s.flags.data_ptr()
        io.pop_ids, io.nonpop_ids, io.counts = s.pop.data_ptr(), s.nonpop.data_ptr(), s.counts.data_ptr()
        io.cold_ids, io.n_cold = s.cold_ids.data_ptr(), s.n_cold.data_ptr()
        io.w_host, io.w_hot, io.staging, io.staging_cap = (
            self.table.dev, self.w_hot.data_ptr(), s.staging.data_ptr(), self.staging_cap)
        io.out, io.workspace, io.ws_bytes = self.out.data_ptr(), s.ws.data_ptr(), s.ws.numel()
        io.write_back = int(self.writeback)
        io.step_flags = flags
        return io

    def plan(self, b: DevBatch, untied=False, handover_kernels=False):
        """Look-ahead segregation of batch b (hl_pipeline_plan): its dispatch,
        cold plan and grouping run on the pipeline's plan stream while the steps
        enqueued before it train; the step of b skips them.  Up to n_sets - 1
        plans ahead of the steps.  handover_kernels: as in step()."""
        if len(self._pending) >= self.n_sets - 1:
            raise RuntimeError(f"{len(self._pending)} look-ahead plans are already pending")
        p = self._par
        self._par = (p + 1) % self.n_sets
        flags = (hl.HL_STEP_UNTIED if untied else 0) | (hl.HL_STEP_HANDOVER_KERNELS if handover_kernels else 0)
        io = self._fill_io(hl.StepIO(), b, self._sets[p], 0.0, flags)
        hl.hl_pipeline_plan(self.pipe, io, torch.cuda.current_stream(self.device))
        self._pending.append((b, p))

    # ------------------------------------------------------------------ learning phase
    def learn(self, prof_batches, k: int | None = None, reset=True):
        for b in prof_batches:
            hl.hl_lookup_gids(self.h, b.rows, b.bag_ptr, b.n_bags, self.gids)
            hl.hl_profile_count(self.h, self.gids, b.n_lookups)
        self.n_hot = hl.hl_profile_topk(self.h, self.k_cap if k is None else k, self.hot_ids, reset_counts=reset)
        hl.hl_hot_fill(self.h, self.hot_ids, self.table.dev, self.w_hot)
        return self.n_hot

    def relearn(self, batches, k: int | None = None):
        """The learning phase again (Sec. V-B: the accelerator switches back to
        learning from time to time; Sec. VI: twice per epoch): access counts
        over `batches` (a sample of recent mini-batches), a new top-K hot set,
        and the hot cache migrated to it (hl_hot_migrate: rows that leave go
        back to the host table, rows that stay keep their trained values, rows
        that enter come from the host table).  Waits for the steps enqueued
        before it; refused while look-ahead plans are pending (they were made
        with the current hot set).  Without write-back the host table holds no
        cold-row updates, so rows that enter carry none either.  Returns the
        new hot-set size."""
        if self._pending:
            raise RuntimeError("look-ahead plans made with the current hot set are pending: step them first")
        self.sync()
        n_old = self.n_hot
        old = self.hot_ids[:n_old].clone()
        w_old = self.w_hot[:n_old].clone()
        for b in batches:
            hl.hl_lookup_gids(self.h, b.rows, b.bag_ptr, b.n_bags, self.gids)
            hl.hl_profile_count(self.h, self.gids, b.n_lookups)
        self.n_hot = hl.hl_profile_topk(self.h, self.k_cap if k is None else k, self.hot_ids, reset_counts=True)
        hl.hl_hot_migrate(self.h, old, n_old, self.hot_ids, w_old, self.w_hot, self.table.dev)
        return self.n_hot

    def set_hot(self, hot_ids: torch.Tensor):
        n = int(hot_ids.numel())
        self.hot_ids[:n].copy_(hot_ids)
        hl.hl_set_hot(self.h, self.hot_ids, n)
        self.n_hot = n
        hl.hl_hot_fill(self.h, self.hot_ids, self.table.dev, self.w_hot)

    # ------------------------------------------------------------------ one mini-batch
    def step(self, b: DevBatch, lr: float | None = None, events=None, mode: str = "pipelined", split_fwd=True,
             untied=False, next=None, handover_kernels=False):
        """classify -> partition -> remap -> cold gather (non-popular) -> forward of
        both mu-batches -> one coalesced SGD step [-> write-back of the cold rows].

        mode "pipelined": the three-stream schedule of the module docstring,
          enqueued by the native pipeline (hl_pipeline_step).  untied: no
          ordering with the current stream (inputs already resident; call
          sync() before using the results).  next: the following batch, or
          a list of the following batches, planned ahead (plan()) up to
          n_sets - 1 of them, to run while this step trains; their own steps
          find them done.  handover_kernels: the handovers between the
          streams as kernels of their own (HL_STEP_HANDOVER_KERNELS), so that
          the path's kernels hold no waits.
        mode "sequential": the fused calls in order on the current stream;
          `events`: optional list of len(STAGES)+1 torch.cuda.Event recorded
          around the stages.
        mode "fwdbwd": as pipelined, but the fetch is awaited before the
          forward/backward section, which `events` (two events) brackets."""
        if mode not in MODES:
            raise ValueError(mode)
        lr = self.w.lr if lr is None else lr
        B, bps, L = b.n_samples, b.bps, b.n_lookups
        if next is not None and mode != "pipelined":
            raise ValueError("look-ahead needs the native pipelined step")
        if mode == "sequential":
            return self._step_sequential(b, lr, events, split_fwd)
        caller = torch.cuda.current_stream(self.device)
        capturing = torch.cuda.is_current_stream_capturing()
        if mode == "fwdbwd" or capturing:  # the Python rendering of the schedule (a graph keeps no CU mask)
            if next is not None:
                raise ValueError("no look-ahead under capture")
            return self._step_pipelined(b, lr, events, mode, caller, capturing)
        flags = (hl.HL_STEP_UNTIED if untied else 0) | (hl.HL_STEP_HANDOVER_KERNELS if handover_kernels else 0)
        nexts = [] if next is None else (list(next) if isinstance(next, (list, tuple)) else [next])
        if nexts and not self._pending:
            self.plan(b, untied, handover_kernels)
        if self._pending:
            if self._pending[0][0] is not b:
                raise RuntimeError("steps must take the batches in the order they were planned")
            _, p = self._pending.pop(0)
            self._use(p)
            flags |= hl.HL_STEP_PLANNED
        else:
            p = self._next_set()
        hl.hl_pipeline_step(self.pipe, self._fill_io(self.io, b, self._sets[p], lr, flags), caller)
        # the next plans after this step: a plan waits only for the steps that
        # used its own buffers, and this step's end signal rides on the next step
        for nb in nexts:
            if len(self._pending) >= self.n_sets - 1:
                break
            if not any(nb is pb for pb, _ in self._pending):
                self.plan(nb, untied, handover_kernels)

    def sync(self, stream=None):
        """The stream (default: current) waits for every step enqueued so far."""
        hl.hl_pipeline_sync(self.pipe, torch.cuda.current_stream(self.device) if stream is None else stream)

    def _step_pipelined(self, b, lr, events, mode, main, capturing):
        h, w = self.h, self.w
        B, bps, L = b.n_samples, b.bps, b.n_lookups
        p = self._next_set()
        cold, ncold = self.cold_ids, self.n_cold
        hl.hl_dispatch(h, b.rows, b.bag_ptr, B, bps, L, self.gids, self.codes, self.flags, self.pop, self.nonpop,
                       self.counts, self.ws)
        if self.writeback and not capturing:
            main.wait_event(self.ev_wb[p])  # the write-back two steps ago read this list
        # a cold lookup makes its sample non-popular, so the cold lookups of all
        # samples are those of the non-popular mu-batch: no sample list needed
        hl.hl_cold_plan(h, self.gids, self.codes, b.bag_ptr, B, bps, L, None, None, B, self.staging_cap, cold, ncold,
                        self.ws)
        self.ev_plan.record(main)
        # working parameters of the non-popular mu-batch over the host link
        self.s_fetch.wait_event(self.ev_plan)
        hl.hl_cold_fetch(h, cold, ncold, self.staging_cap, self.table.dev, self.staging, stream=self.s_fetch)
        self.ev_fetch.record(self.s_fetch)
        if mode == "fwdbwd":
            main.wait_event(self.ev_fetch)
            if events is not None:
                events[0].record(main)
        # the backward's grouping needs only the codes
        self.s_group.wait_event(self.ev_fetch if mode == "fwdbwd" else self.ev_plan)
        if b.dY is not None:
            hl.hl_embbag_bwd_plan(h, self.staging_cap, self.codes, b.bag_ptr, B, bps, L, None, None, B, self.ws,
                                  stream=self.s_group)
        # popular mu-batch, and the hot rows of the non-popular one, while the fetch runs
        hl.hl_embbag_fwd_part(h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                              self.pop, self.counts[0:], B, self.out, 0)
        hl.hl_embbag_fwd_part(h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                              self.nonpop, self.counts[1:], B, self.out, 1)
        self.ev_fwdhot.record(main)
        # the backward's reduction and hot-row updates once both forwards have read the hot rows
        self.s_group.wait_event(self.ev_fwdhot)
        if b.dY is not None:
            hl.hl_embbag_bwd_apply_part(h, self.w_hot, self.staging, self.staging_cap, B, bps, L, b.dY, lr, 1,
                                        self.ws, stream=self.s_group)
        self.ev_group.record(self.s_group)
        # the staging rows: cold half of the non-popular forward, then their updates
        main.wait_event(self.ev_fetch)
        hl.hl_embbag_fwd_part(h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                              self.nonpop, self.counts[1:], B, self.out, 2)
        main.wait_event(self.ev_group)
        if b.dY is not None:
            hl.hl_embbag_bwd_apply_part(h, self.w_hot, self.staging, self.staging_cap, B, bps, L, b.dY, lr, 2,
                                        self.ws)
        if mode == "fwdbwd" and events is not None:
            events[1].record(main)
        if self.writeback:
            self.ev_apply.record(main)
            self.s_fetch.wait_event(self.ev_apply)
            hl.hl_cold_scatter(h, cold, ncold, self.staging_cap, self.staging, self.table.dev, stream=self.s_fetch)
            self.ev_wb[p].record(self.s_fetch)
            if capturing:  # a graph joins every stream it forked
                main.wait_event(self.ev_wb[p])

    def capture(self, b: DevBatch, lr: float | None = None):
        """A HIP graph of one pipelined step over batch b (the Python rendering
        of the schedule, on unmasked streams): replaying it runs the whole step
        (all three streams, joined) with one launch.  Run one eager
        step of at least this size first (the cold plan's hash table is
        allocated on first use).  Returns (graph, bufs): bufs holds the
        per-step buffers the graph writes (gids, codes, flags, pop, nonpop,
        counts, cold_ids, n_cold, ws); later eager steps alternate sets."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.step(b, lr=lr, mode="pipelined")
        return g, next(s for s in self._sets if s.codes is self.codes)

    def _step_sequential(self, b, lr, events, split_fwd):
        B, bps, L = b.n_samples, b.bps, b.n_lookups
        ev = events
        p = self._next_set()
        main = torch.cuda.current_stream(self.device)
        if self.writeback:
            main.wait_event(self.ev_wb[p])

        def mark(i):
            if ev is not None:
                ev[i].record()

        mark(0)
        hl.hl_lookup_gids(self.h, b.rows, b.bag_ptr, b.n_bags, self.gids)
        mark(1)
        hl.hl_classify(self.h, self.gids, b.bag_ptr, B, bps, L, self.flags)
        mark(2)
        hl.hl_partition(self.h, self.flags, B, self.pop, self.nonpop, self.counts, self.ws)
        mark(3)
        hl.hl_remap(self.h, self.gids, L, self.codes)
        mark(4)
        hl.hl_cold_gather(self.h, self.gids, self.codes, b.bag_ptr, B, bps, L, self.nonpop, self.counts[1:], B,
                          self.table.dev, self.staging, self.staging_cap, self.cold_ids, self.n_cold, self.ws)
        mark(5)
        if split_fwd:
            hl.hl_embbag_fwd(self.h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                             self.pop, self.counts[0:], B, self.out)
            mark(6)
            hl.hl_embbag_fwd(self.h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                             self.nonpop, self.counts[1:], B, self.out)
        elif b.dY is not None:
            # the forward with the backward's grouping beside it, then the update
            hl.hl_embbag_fwd_plan(self.h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                                  self.out, self.ws)
            mark(6)
        else:
            hl.hl_embbag_fwd(self.h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                             None, None, B, self.out)
            mark(6)
        mark(7)
        if b.dY is not None:
            if split_fwd:
                hl.hl_embbag_bwd_sgd(self.h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B,
                                     bps, L, None, None, B, b.dY, lr, self.ws)
            else:
                hl.hl_embbag_bwd_apply(self.h, self.w_hot, self.staging, self.staging_cap, B, bps, L, b.dY, lr,
                                       self.ws)
        mark(8)
        if self.writeback:
            hl.hl_cold_scatter(self.h, self.cold_ids, self.n_cold, self.staging_cap, self.staging, self.table.dev)
            self.ev_wb[p].record(main)

    def device_error(self):
        return hl.hl_last_device_error(self.h)

    @property
    def s_fetch(self):
        return self._pystreams()[0]

    @property
    def s_group(self):
        return self._pystreams()[1]

    def _pystreams(self):
        """Streams of the Python rendering of the schedule (graph capture and the
        fwd+bwd timing mode), created on first use."""
        if self._py_streams is None:
            self._py_streams = (torch.cuda.Stream(device=self.device), torch.cuda.Stream(device=self.device))
        return self._py_streams

    def close(self):
        torch.cuda.synchronize()
        if self.pipe:
            hl.hl_pipeline_destroy(self.pipe)
            self.pipe = None
        self.h.close()
