"""The five synthetic workloads the hot path is built and measured on.

Each workload stands in for one of the paper's model/dataset shapes (Table
"Recommender Model Architecture and Parameters"): the DLRM-small/large shapes
for the Criteo Kaggle/Terabyte models (26 sparse features, dim 16/64), the
multi-hot shape for the paper's synthetic multi-hot models (Sec. VII-F "Varying
Model Size"), the TBSM shape for the Taobao time-series model (21 time steps,
3 sparse features, dim 16).  The paper's datasets are not available; these are
seeded Zipf stand-ins.

Hot-set size rules (the paper gives a ~512 MB budget for hot embeddings, Sec.
II-B, and a fixed-capacity tracker, Sec. V-B, but no top-K formula): a fraction
of all rows, rounded up, or a byte budget divided by the row size, rounded down
(MB = MiB, GB = GiB).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    n_tables: int
    dim: int
    dtype: str                     # "f32" or "bf16" (storage); pooling accumulates in fp32
    batch: int                     # samples per mini-batch
    steps: int = 1                 # time steps per sample (TBSM); bags/sample = steps * n_tables
    alpha: float = 1.1             # Zipf exponent of the per-table index distribution
    rows_fixed: tuple = ()         # explicit rows per table, or ...
    rows_loguniform: tuple = ()    # ... (lo, hi) for a seeded log-uniform draw per table
    bag_len_poisson: float = 0.0   # >0: multi-hot bags, Poisson(mean) clipped to bag_len_clip
    bag_len_clip: tuple = (1, 64)
    repeat_prob: float = 0.0       # TBSM locality: P(step s repeats step s-1's index)
    hot_frac: float = 0.0          # hot-set size rule: ceil(frac * n_rows) ...
    hot_budget_bytes: int = 0      # ... or floor(budget / row_bytes)
    n_dense: int = 0               # dense features carried with each sample (unused by kernels)
    lr: float = 0.01
    profile_batches: int = 16
    measured_batches: int = 32
    seed: int = 0

    @property
    def bags_per_sample(self) -> int:
        return self.steps * self.n_tables

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def row_bytes(self) -> int:
        return self.dim * self.elem_bytes

    def k_cap(self, n_rows: int) -> int:
        if self.hot_budget_bytes:
            return self.hot_budget_bytes // self.row_bytes
        return int(math.ceil(self.hot_frac * n_rows - 1e-9))


MiB = 1 << 20
GiB = 1 << 30

WORKLOADS = {
    "tiny": Workload(
        name="tiny", n_tables=8, dim=16, dtype="f32", batch=1024, alpha=1.05,
        rows_fixed=(10_000,) * 8, hot_frac=0.01, seed=1001),
    "dlrm-small": Workload(
        name="dlrm-small", n_tables=26, dim=16, dtype="f32", batch=4096, alpha=1.1,
        rows_loguniform=(10, 10_000_000), hot_budget_bytes=512 * MiB, n_dense=13, seed=1002),
    "dlrm-large": Workload(
        name="dlrm-large", n_tables=26, dim=64, dtype="f32", batch=8192, alpha=1.1,
        rows_loguniform=(100, 40_000_000), hot_budget_bytes=4 * GiB, seed=1003),
    "multi-hot": Workload(
        name="multi-hot", n_tables=8, dim=128, dtype="bf16", batch=2048, alpha=1.2,
        rows_fixed=(5_000_000,) * 8, bag_len_poisson=20.0, bag_len_clip=(1, 64),
        hot_frac=0.02, seed=1004),
    "tbsm": Workload(
        name="tbsm", n_tables=3, dim=16, dtype="f32", batch=1024, steps=21, alpha=1.2,
        rows_fixed=(1_000_000, 100_000, 10_000), repeat_prob=0.7, hot_frac=0.01, seed=1005),
}

ORDER = ["tiny", "dlrm-small", "dlrm-large", "multi-hot", "tbsm"]


def scaled(w: Workload, *, batch: int | None = None, row_scale: float | None = None,
           max_rows: int | None = None, name: str | None = None, **kw) -> Workload:
    """A smaller copy of a workload for oracle-speed parity runs (same structure)."""
    d = dict(w.__dict__)
    if batch is not None:
        d["batch"] = batch
    if row_scale is not None or max_rows is not None:
        if w.rows_fixed:
            rows = [max(1, int(r * (row_scale or 1.0))) for r in w.rows_fixed]
            if max_rows:
                rows = [min(r, max_rows) for r in rows]
            d["rows_fixed"] = tuple(rows)
        else:
            lo, hi = w.rows_loguniform
            hi2 = int(hi * (row_scale or 1.0))
            if max_rows:
                hi2 = min(hi2, max_rows)
            d["rows_loguniform"] = (min(lo, hi2), max(hi2, 1))
    if w.hot_budget_bytes and row_scale is not None:
        d["hot_budget_bytes"] = max(w.row_bytes, int(w.hot_budget_bytes * row_scale))
    d["name"] = name or (w.name + "-scaled")
    d.update(kw)
    return Workload(**d)
