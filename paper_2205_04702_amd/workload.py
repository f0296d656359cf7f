"""Seeded synthetic inputs for embedding-layer training runs.

This module only draws numbers: table contents, sparse-ID batches and upstream
gradients.  It holds none of the training or caching arithmetic, so both the
GPU path and the CPU oracle can be fed from it.

The paper trains on traces synthesised from real-dataset access distributions
(Methodology, "Benchmarks"); those datasets are not available here, so Zipf and
uniform ID distributions over a seed-shuffled row order stand in for them.

Every stream is keyed by (seed, purpose, table, step) through numpy's
SeedSequence, so any batch can be regenerated on its own, in any order.
"""
from __future__ import annotations

import dataclasses
import math
from functools import lru_cache

import numpy as np

_INIT, _IDS, _GRAD, _PERM, _MIXED = 1, 2, 3, 4, 5


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape of one synthetic embedding-training workload."""

    name: str
    rows: tuple            # rows per table
    dim: int               # embedding dimension (fp32)
    batch: int             # samples per mini-batch (= bags per table)
    pooling: tuple         # IDs per bag, per table
    dist: tuple            # per table: ("uniform",) or ("zipf", alpha)
    slots: tuple           # scratchpad slots per table
    lookahead: int         # successor batches visible to the planner
    steps: int
    lr: float = 0.01
    grad_sigma: float = 1.0
    seed: int = 0

    @property
    def tables(self) -> int:
        return len(self.rows)

    @property
    def nnz(self) -> int:
        return self.batch * int(sum(self.pooling))

    def ids_per_table(self) -> list:
        return [self.batch * p for p in self.pooling]

    def describe(self) -> dict:
        return {
            "workload": self.name,
            "tables": self.tables,
            "rows": (list(self.rows) if len(set(self.rows)) > 1 else int(self.rows[0])),
            "dim": self.dim,
            "batch": self.batch,
            "pooling": (list(self.pooling) if len(set(self.pooling)) > 1 else int(self.pooling[0])),
            "slots": (list(self.slots) if len(set(self.slots)) > 1 else int(self.slots[0])),
            "lookahead": self.lookahead,
            "steps": self.steps,
            "lr": self.lr,
            "grad_sigma": self.grad_sigma,
            "dist": sorted({d[0] if d[0] == "uniform" else f"zipf{d[1]}" for d in self.dist}),
        }


def _uniform_tables(n, rows, dim, batch, pooling, dist, slots, lookahead, steps, name,
                    sigma=1.0):
    return Workload(name=name, rows=(rows,) * n, dim=dim, batch=batch, pooling=(pooling,) * n,
                    dist=(dist,) * n, slots=(slots,) * n, lookahead=lookahead, steps=steps,
                    grad_sigma=sigma)


def mixed_workload(seed: int = 0, budget_bytes: float = 40e9, steps: int = 200) -> Workload:
    """64 tables, rows log-uniform in [1e3, 2e7], D=64, B=8192, pooling U[1,80];
    tables 0..31 draw uniform IDs, 32..63 Zipf(1.2); the scratchpad budget is
    split by first guaranteeing one window's worth of IDs per table and then
    water-filling the rest in proportion to table size (capped at the table)."""
    rng = np.random.default_rng([seed, _MIXED])
    T, D, B, L = 64, 64, 8192, 6
    rows = np.floor(np.exp(rng.uniform(math.log(1e3), math.log(2e7), size=T))).astype(np.int64)
    pooling = rng.integers(1, 81, size=T)
    dist = tuple(("uniform",) if t < 32 else ("zipf", 1.2) for t in range(T))
    total_rows = int(budget_bytes // (4 * D))
    base = np.minimum(rows, (L + 1) * B * pooling)
    slots = base.astype(np.float64)
    remaining = total_rows - base.sum()
    free = rows - base
    # water-fill the remaining budget proportionally to table size, capped at the table
    while remaining > 0.5 and free.sum() > 0:
        share = remaining * rows * (free > 0) / max(1, (rows * (free > 0)).sum())
        add = np.minimum(share, free)
        slots += add
        free = free - add
        remaining -= add.sum()
        if add.sum() < 0.5:
            break
    slots = np.minimum(np.floor(slots).astype(np.int64), rows)
    return Workload(name="mixed-64t-d64", rows=tuple(int(r) for r in rows), dim=D, batch=B,
                    pooling=tuple(int(p) for p in pooling), dist=dist,
                    slots=tuple(int(s) for s in slots), lookahead=L, steps=steps, seed=seed)


def get_workload(name: str) -> Workload:
    """The named synthetic workloads (sizes follow the benchmark configurations)."""
    if name == "tiny":
        return _uniform_tables(4, 20_000, 32, 128, 4, ("uniform",), 2_048, 2, 50,
                               "tiny-4x20k-d32")
    if name == "zipf-8x1M":
        return _uniform_tables(8, 1_000_000, 64, 1_024, 8, ("zipf", 1.05), 100_000, 3, 200,
                               "zipf-8x1M-d64")
    if name == "zipf-26x4M":
        return _uniform_tables(26, 4_000_000, 128, 2_048, 20, ("zipf", 1.1), 200_000, 4, 500,
                               "zipf-26x4M-d128", sigma=0.1)
    if name == "zipf-26x10M":
        return _uniform_tables(26, 10_000_000, 128, 4_096, 40, ("zipf", 0.9), 200_000, 4, 300,
                               "zipf-26x10M-d128")
    if name == "mixed":
        return mixed_workload()
    raise KeyError(name)


WORKLOADS = ("tiny", "zipf-8x1M", "zipf-26x4M", "zipf-26x10M", "mixed")


def custom(rows, dim, batch, pooling, slots, lookahead, steps, dist=("uniform",), seed=0,
           lr=0.01, sigma=1.0, name="custom") -> Workload:
    """Small ad-hoc workloads for tests; scalars broadcast over tables."""
    T = len(rows) if isinstance(rows, (list, tuple)) else 1
    def per_table(x):
        if isinstance(x, (list, tuple)) and len(x) == T and not isinstance(x[0], str):
            return tuple(x)
        return (x,) * T
    rows_t = per_table(rows)
    T = len(rows_t)
    dists = dist if (isinstance(dist, tuple) and len(dist) == T and isinstance(dist[0], tuple)) \
        else (dist,) * T
    return Workload(name=name, rows=tuple(int(r) for r in rows_t), dim=dim, batch=batch,
                    pooling=tuple(int(p) for p in per_table(pooling)), dist=tuple(dists),
                    slots=tuple(int(s) for s in per_table(slots)), lookahead=lookahead,
                    steps=steps, seed=seed, lr=lr, grad_sigma=sigma)


# ----------------------------------------------------------------------------- draws

@lru_cache(maxsize=8)
def _zipf_cdf(rows: int, alpha: float) -> np.ndarray:
    """Cumulative probabilities of P(rank k) proportional to k^-alpha, k = 1..rows (fp64)."""
    w = np.arange(1, rows + 1, dtype=np.float64) ** (-alpha)
    c = np.cumsum(w)
    c /= c[-1]
    return c


@lru_cache(maxsize=128)
def _row_permutation(seed: int, table: int, rows: int) -> np.ndarray:
    return np.random.default_rng([seed, _PERM, table]).permutation(rows).astype(np.int32)


def table_ids(w: Workload, t: int, step: int, n: int | None = None) -> np.ndarray:
    """Sparse row IDs of table t in mini-batch `step` (int32, i.i.d. per draw)."""
    R = w.rows[t]
    n = w.batch * w.pooling[t] if n is None else n
    rng = np.random.default_rng([w.seed, _IDS, t, step])
    d = w.dist[t]
    if d[0] == "uniform":
        return rng.integers(0, R, size=n, dtype=np.int64).astype(np.int32)
    if d[0] == "zipf":
        u = rng.random(n)
        k = np.searchsorted(_zipf_cdf(R, float(d[1])), u, side="right")
        np.minimum(k, R - 1, out=k)
        return _row_permutation(w.seed, t, R)[k]
    raise ValueError(d)


def fixed_offsets(batch: int, pooling) -> np.ndarray:
    """CSR bag offsets [T*B+1] for a fixed number of IDs per bag per table."""
    lens = np.repeat(np.asarray(pooling, dtype=np.int64), batch)
    off = np.zeros(lens.size + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    return off.astype(np.int32)


def batch(w: Workload, step: int):
    """One mini-batch in table-major CSR form.

    Returns (ids, bag_off): ids is int32 [NNZ] with table 0's IDs first, then
    table 1's, ...; bag_off is int32 [T*B+1] and bag g = t*B + b spans
    ids[bag_off[g]:bag_off[g+1]] (row numbers local to table t).
    """
    ids = np.concatenate([table_ids(w, t, step) for t in range(w.tables)])
    return ids, fixed_offsets(w.batch, w.pooling)


def ragged_batch(w: Workload, step: int, max_len: int, empty_frac: float = 0.1):
    """A mini-batch with per-bag lengths drawn in [0, max_len] (some bags empty)."""
    rng = np.random.default_rng([w.seed, _IDS, 1000, step])
    T, B = w.tables, w.batch
    lens = rng.integers(1, max_len + 1, size=T * B)
    lens[rng.random(T * B) < empty_frac] = 0
    off = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    parts = []
    for t in range(T):
        n = int(off[(t + 1) * B] - off[t * B])
        parts.append(table_ids(w, t, step, n=n) if n else np.zeros(0, np.int32))
    return np.concatenate(parts).astype(np.int32), off.astype(np.int32)


def thinned_batch(w: Workload, step: int, tables=None, max_ids: int | None = None):
    """batch(w, step) with only the IDs of `tables` kept (the bags of the other
    tables become empty; () gives a batch without any ID), then only the first
    `max_ids` of those, in CSR order (later bags empty)."""
    ids, off = batch(w, step)
    B = w.batch
    lens = np.diff(off.astype(np.int64))
    if tables is not None:
        for t in range(w.tables):
            if t not in tables:
                lens[t * B:(t + 1) * B] = 0
    if max_ids is not None:
        lens = np.minimum(lens, np.maximum(max_ids - (np.cumsum(lens) - lens), 0))
    keep = np.zeros(ids.size, dtype=bool)
    for g in np.nonzero(lens)[0]:
        keep[int(off[g]):int(off[g]) + int(lens[g])] = True
    new_off = np.zeros(lens.size + 1, dtype=np.int64)
    np.cumsum(lens, out=new_off[1:])
    return ids[keep].astype(np.int32), new_off.astype(np.int32)


def grads(w: Workload, step: int) -> np.ndarray:
    """Upstream gradient of the pooled outputs, float32 [T, B, D], N(0, sigma^2)."""
    rng = np.random.default_rng([w.seed, _GRAD, step])
    g = rng.standard_normal((w.tables, w.batch, w.dim), dtype=np.float32)
    if w.grad_sigma != 1.0:
        g *= np.float32(w.grad_sigma)
    return g


def init_table(w: Workload, t: int, out: np.ndarray | None = None) -> np.ndarray:
    """Initial weights of table t: U[-0.05, 0.05) in fp32, written into `out` if given."""
    shape = (w.rows[t], w.dim)
    if out is None:
        out = np.empty(shape, dtype=np.float32)
    assert out.shape == shape and out.dtype == np.float32
    rng = np.random.default_rng([w.seed, _INIT, t])
    rng.random(out=out.reshape(-1), dtype=np.float32)
    out *= np.float32(0.1)
    out -= np.float32(0.05)
    return out


def window(u: int, lookahead: int, steps: int) -> list:
    """Indices of the batches visible when batch u is planned: u .. u+L, cut at the end."""
    return list(range(u, min(u + lookahead, steps - 1) + 1))
