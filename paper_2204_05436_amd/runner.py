"""Orchestration of the hot path on one GPU: device buffers for a workload and
the library calls in the order the paper's pipeline runs them (Sec. IV: the
learning phase, then per mini-batch classification, fragmentation into the
popular and non-popular mu-batches, working-parameter gather for the
non-popular one, forward of both, and the update).  No arithmetic here: every
step is a call into libhotline."""
from __future__ import annotations

from dataclasses import dataclass

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


class HotPath:
    def __init__(self, w: Workload, rows_per_table, table: hl.HostTable, max_lookups: int, max_samples: int,
                 device="cuda", k_cap: int | None = None, staging_cap: int | None = None):
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
        self.ws = torch.zeros(wsb, dtype=torch.uint8, device=device)
        sdt = torch.float32 if w.dtype == "f32" else torch.int16
        self.sdt = sdt
        self.w_hot = torch.zeros((self.k_cap, w.dim), dtype=sdt, device=device)
        self.staging_cap = int(staging_cap if staging_cap is not None else max(1, self.max_lookups))
        self.staging = torch.zeros((self.staging_cap, w.dim), dtype=sdt, device=device)
        self.hot_ids = torch.zeros(max(1, min(self.k_cap, n_rows)), dtype=torch.int32, device=device)
        L, B = max(1, self.max_lookups), max(1, self.max_samples)
        i32 = dict(dtype=torch.int32, device=device)
        self.gids = torch.zeros(L, **i32)
        self.codes = torch.zeros(L, **i32)
        self.flags = torch.zeros(B, dtype=torch.uint8, device=device)
        self.pop = torch.zeros(B, **i32)
        self.nonpop = torch.zeros(B, **i32)
        self.counts = torch.zeros(2, **i32)
        self.cold_ids = torch.zeros(self.staging_cap, **i32)
        self.n_cold = torch.zeros(1, **i32)
        self.out = torch.zeros((max(1, max_bags), w.dim), dtype=torch.float32, device=device)
        self.n_hot = 0

    # ------------------------------------------------------------------ learning phase
    def learn(self, prof_batches, k: int | None = None, reset=True):
        for b in prof_batches:
            hl.hl_lookup_gids(self.h, b.rows, b.bag_ptr, b.n_bags, self.gids)
            hl.hl_profile_count(self.h, self.gids, b.n_lookups)
        self.n_hot = hl.hl_profile_topk(self.h, self.k_cap if k is None else k, self.hot_ids, reset_counts=reset)
        hl.hl_hot_fill(self.h, self.hot_ids, self.table.dev, self.w_hot)
        return self.n_hot

    def set_hot(self, hot_ids: torch.Tensor):
        n = int(hot_ids.numel())
        self.hot_ids[:n].copy_(hot_ids)
        hl.hl_set_hot(self.h, self.hot_ids, n)
        self.n_hot = n
        hl.hl_hot_fill(self.h, self.hot_ids, self.table.dev, self.w_hot)

    # ------------------------------------------------------------------ one mini-batch
    def step(self, b: DevBatch, lr: float | None = None, events=None, split_fwd=True):
        """classify -> partition -> remap -> cold gather (non-popular) -> forward of
        both mu-batches -> one coalesced SGD step.  `events`: optional list of
        len(STAGES)+1 torch.cuda.Event recorded around the stages."""
        lr = self.w.lr if lr is None else lr
        B, bps, L = b.n_samples, b.bps, b.n_lookups
        ev = events

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
        else:
            hl.hl_embbag_fwd(self.h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                             None, None, B, self.out)
            mark(6)
        mark(7)
        if b.dY is not None:
            hl.hl_embbag_bwd_sgd(self.h, self.w_hot, self.staging, self.staging_cap, self.codes, b.bag_ptr, B, bps, L,
                                 None, None, B, b.dY, lr, self.ws)
        mark(8)

    def device_error(self):
        return hl.hl_last_device_error(self.h)

    def close(self):
        self.h.close()
