"""Seeded synthetic inputs for one sparse-embedding training step.

This module only draws random numbers and lays them out; it holds none of the
Tensor Casting arithmetic (no gather, reduce, sort, coalesce or update). Both
the CPU oracle side and the HIP side take their inputs from here.

What a workload is (paper Sec. II-B, the embedding gather-reduce problem):
``num_tables`` tables of ``rows_per_table`` fp32 rows of width ``dim``; every
table is pooled over ``batch`` bags; each bag gathers a list of row ids. The
index array is kept in bag-major CSR form: ``indices`` holds table-local row
ids, ``bag_offsets[g]..bag_offsets[g+1]`` are the pairs of bag
``g = t * batch + b``, and ``table_row_offset[t]`` is the first global row of
table ``t`` in the concatenated table.

The datasets whose lookup skew the paper measured (Sec. III-B) are not
available here, so bounded Zipf and uniform index streams stand in for them.

Random streams: ``numpy.random.Generator(PCG64(SeedSequence([seed, cfg, stream,
table, step])))`` with stream ids 1 = row permutation, 2 = indices,
3 = pooling lengths, 4 = output gradient.

Table values come from a counter-based generator, SplitMix64 (Steele, Lea and
Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014), so any
row can be regenerated on its own: the value of element ``e`` of the
concatenated table (``e = global_row * dim + col``) is the ``(e+1)``-th output of
SplitMix64 started from state ``seed``, i.e. ``mix(seed + (e+1) * GOLDEN)``;
its top 24 bits give ``u in [0, 1)`` and the fp32 value is ``lo + (hi-lo)*u``,
two separately rounded fp32 operations.
"""
from __future__ import annotations

import dataclasses
import functools

import numpy as np

# SplitMix64 constants, from the published definition.
SM64_GOLDEN = 0x9E3779B97F4A7C15
SM64_MUL1 = 0xBF58476D1CE4E5B9
SM64_MUL2 = 0x94D049BB133111EB

STREAM_PERM, STREAM_INDEX, STREAM_POOL, STREAM_GRAD = 1, 2, 3, 4


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic embedding-training workload."""

    name: str
    cfg_id: int
    num_tables: int
    rows_per_table: int
    dim: int
    batch: int                 # bags per table
    pooling: str               # "fixed" | "poisson"
    pooling_value: int         # fixed length, or Poisson mean (min length 1)
    dist: str                  # "uniform" | "zipf"
    alpha: float = 0.0         # Zipf exponent
    optimizer: str = "sgd"     # "sgd" | "adagrad" | "rmsprop" | "rowwise_adagrad"
    lr: float = 0.01
    eps: float = 1e-8
    gamma: float = 0.99        # RMSprop decay (Eq. 1)
    init_lo: float = -0.01
    init_hi: float = 0.01

    @property
    def num_bags(self) -> int:
        return self.num_tables * self.batch

    @property
    def total_rows(self) -> int:
        return self.num_tables * self.rows_per_table

    def scaled(self, *, name=None, num_tables=None, rows_per_table=None,
               dim=None, batch=None, pooling_value=None, optimizer=None) -> "Workload":
        """The same distributions at a smaller (or different) shape, optionally
        with another optimizer."""
        return dataclasses.replace(
            self,
            optimizer=optimizer or self.optimizer,
            name=name or (self.name + "-scaled"),
            num_tables=num_tables or self.num_tables,
            rows_per_table=rows_per_table or self.rows_per_table,
            dim=dim or self.dim,
            batch=batch or self.batch,
            pooling_value=pooling_value or self.pooling_value,
        )


def variant(w: Workload, *, batch=None, dim=None, optimizer=None) -> Workload:
    """w with another batch size, dimension or optimizer (w itself if none
    changes), renamed to match: the name's -d, -b and optimizer fields."""
    if ((batch is None or batch == w.batch) and (dim is None or dim == w.dim)
            and (optimizer is None or optimizer == w.optimizer)):
        return w
    parts = w.name.split("-")
    batch, dim, optimizer = batch or w.batch, dim or w.dim, optimizer or w.optimizer
    parts = [f"d{dim}" if p == f"d{w.dim}" else f"b{batch}" if p == f"b{w.batch}" else p
             for p in parts[:-1]] + [optimizer]
    return dataclasses.replace(w, name="-".join(parts), batch=batch, dim=dim,
                               optimizer=optimizer)


# The five workloads of the measurement plan, named by what they are.
WORKLOADS = {
    "c1": Workload("1x100k-d64-b256-pool20-uniform-sgd", 0, 1, 100_000, 64, 256,
                   "fixed", 20, "uniform", optimizer="sgd"),
    "c2": Workload("8x1M-d64-b2048-pool80-zipf1.05-sgd", 1, 8, 1_000_000, 64, 2048,
                   "fixed", 80, "zipf", 1.05, optimizer="sgd"),
    "c3": Workload("8x5M-d128-b4096-poisson40-zipf1.2-adagrad", 2, 8, 5_000_000, 128, 4096,
                   "poisson", 40, "zipf", 1.2, optimizer="adagrad"),
    "c4": Workload("32x1M-d256-b8192-pool20-uniform-sgd", 3, 32, 1_000_000, 256, 8192,
                   "fixed", 20, "uniform", optimizer="sgd"),
    "c5": Workload("1x50M-d128-b16384-pool100-zipf0.9-adagrad", 4, 1, 50_000_000, 128, 16384,
                   "fixed", 100, "zipf", 0.9, optimizer="adagrad"),
}


@dataclasses.dataclass
class Batch:
    """One step's sparse input and output gradient (host arrays)."""

    indices: np.ndarray           # int32 [N], table-local row ids
    bag_offsets: np.ndarray       # int32 [T*B + 1]
    table_row_offset: np.ndarray  # int64 [T + 1]
    grad_out: np.ndarray          # float32 [T*B, D]

    @property
    def num_pairs(self) -> int:
        return int(self.bag_offsets[-1])


def _rng(seed: int, cfg: int, stream: int, table: int, step: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [seed, cfg, stream, table, step])))


@functools.lru_cache(maxsize=8)
def _zipf_cdf(rows: int, alpha: float) -> np.ndarray:
    """Unnormalised cumulative weights of ranks 1..rows under k^-alpha (float64)."""
    k = np.arange(1, rows + 1, dtype=np.float64)
    return np.cumsum(k ** (-alpha))


@functools.lru_cache(maxsize=64)
def _row_permutation(seed: int, cfg: int, table: int, rows: int) -> np.ndarray:
    """Random map from Zipf rank to row id, fixed per table across steps."""
    return _rng(seed, cfg, STREAM_PERM, table, 0).permutation(rows).astype(np.int32)


def draw_table_indices(w: Workload, table: int, count: int, step: int, seed: int = 0) -> np.ndarray:
    """``count`` i.i.d. row ids of one table (int32)."""
    rng = _rng(seed, w.cfg_id, STREAM_INDEX, table, step)
    if w.dist == "uniform":
        return rng.integers(0, w.rows_per_table, size=count, dtype=np.int64).astype(np.int32)
    if w.dist == "zipf":
        cdf = _zipf_cdf(w.rows_per_table, float(w.alpha))
        u = rng.random(count) * cdf[-1]
        rank = np.minimum(np.searchsorted(cdf, u, side="right"), w.rows_per_table - 1)
        return _row_permutation(seed, w.cfg_id, table, w.rows_per_table)[rank]
    raise ValueError(f"unknown index distribution {w.dist!r}")


def draw_pooling(w: Workload, table: int, step: int, seed: int = 0) -> np.ndarray:
    """Bag lengths of one table (int64 [B])."""
    if w.pooling == "fixed":
        return np.full(w.batch, w.pooling_value, dtype=np.int64)
    if w.pooling == "poisson":
        rng = _rng(seed, w.cfg_id, STREAM_POOL, table, step)
        return np.maximum(1, rng.poisson(w.pooling_value, size=w.batch)).astype(np.int64)
    raise ValueError(f"unknown pooling {w.pooling!r}")


def table_row_offsets(w: Workload) -> np.ndarray:
    return (np.arange(w.num_tables + 1, dtype=np.int64) * w.rows_per_table)


def make_batch(w: Workload, step: int = 0, seed: int = 0, with_grad: bool = True) -> Batch:
    """Bag-major CSR index array plus an N(0,1) fp32 output gradient."""
    lengths, idx = [], []
    for t in range(w.num_tables):
        ln = draw_pooling(w, t, step, seed)
        lengths.append(ln)
        idx.append(draw_table_indices(w, t, int(ln.sum()), step, seed))
    lengths = np.concatenate(lengths)
    offsets = np.zeros(w.num_bags + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    if offsets[-1] >= 2 ** 31:
        raise ValueError("more than 2^31-1 pairs")
    if with_grad:
        grad = _rng(seed, w.cfg_id, STREAM_GRAD, 0, step).standard_normal(
            (w.num_bags, w.dim), dtype=np.float32)
    else:
        grad = np.zeros((0, w.dim), dtype=np.float32)
    return Batch(np.concatenate(idx).astype(np.int32), offsets.astype(np.int32),
                 table_row_offsets(w), grad)


def splitmix64_at(state0: int, counters: np.ndarray) -> np.ndarray:
    """Outputs number ``counters`` (1-based) of SplitMix64 started at ``state0``."""
    with np.errstate(over="ignore"):
        z = np.uint64(state0 & 0xFFFFFFFFFFFFFFFF) + counters.astype(np.uint64) * np.uint64(SM64_GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(SM64_MUL1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(SM64_MUL2)
        return z ^ (z >> np.uint64(31))


def table_rows(w: Workload, global_rows: np.ndarray, seed: int = 0) -> np.ndarray:
    """Initial fp32 values of the given global rows, ``[len(rows), dim]``."""
    rows = np.asarray(global_rows, dtype=np.int64)
    e = rows[:, None] * np.int64(w.dim) + np.arange(w.dim, dtype=np.int64)[None, :]
    x = splitmix64_at(seed, (e + 1).astype(np.uint64))
    u = (x >> np.uint64(40)).astype(np.float32) * np.float32(2.0 ** -24)
    lo, hi = np.float32(w.init_lo), np.float32(w.init_hi)
    span = np.float32(hi - lo)
    return (lo + span * u).astype(np.float32)
