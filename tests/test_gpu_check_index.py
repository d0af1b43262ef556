"""tc_check_index on the GPU: the first problem of an index array (lowest
kind, then lowest position), against the layout's definition written out
in numpy below, on valid workloads, planted errors and random corruptions.
Exact integer comparison."""
import numpy as np
import pytest
import torch

from paper_2010_13100_amd import tc
from paper_2010_13100_amd import workload as wl

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda", 0)
OK = (tc.TC_INDEX_OK, -1)


def expected(off, bo, idx, T, B, total_rows, bound):
    """The definition: table offsets, then bag offsets, then indices."""
    n = len(idx)
    bad_t = [t for t in range(T + 1)
             if (t == 0 and off[0] != 0) or (t > 0 and off[t] < off[t - 1])
             or (t == T and off[T] != total_rows)]
    if bad_t:
        return (tc.TC_INDEX_BAD_TABLE_OFFSETS, bad_t[0])
    d = np.diff(bo.astype(np.int64))
    bad_g = sorted(([0] if bo[0] != 0 else []) + (np.nonzero(d < 0)[0] + 1).tolist()
                   + ([T * B] if bo[T * B] != n else []))
    if bad_g:
        return (tc.TC_INDEX_BAD_BAG_OFFSETS, bad_g[0])
    if T == 0 or n == 0:
        return OK
    starts = bo[np.arange(T, dtype=np.int64) * B]
    t_of = np.searchsorted(starts, np.arange(n), side="right") - 1
    rows = (off[1:] - off[:-1])[t_of]
    i = idx.astype(np.int64)
    bad = (i < 0) | (i >= rows) | ((bound > 0) & (i >= bound))
    j = np.nonzero(bad)[0]
    return (tc.TC_INDEX_OUT_OF_RANGE, int(j[0])) if len(j) else OK


def run(off, bo, idx, T, B, total_rows, bound, report=None):
    n = len(idx)
    report = report if report is not None else torch.full((2,), 77, dtype=torch.int64,
                                                          device=DEV)
    d_idx = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(DEV) if n else None
    tc.tc_check_index(torch.from_numpy(np.ascontiguousarray(off, np.int64)).to(DEV), T, B,
                      total_rows, bound, d_idx,
                      torch.from_numpy(np.ascontiguousarray(bo, np.int32)).to(DEV), n, report)
    torch.cuda.synchronize()
    r = report.cpu().tolist()
    return (r[0], r[1])


def layout(seed, T=5, B=7, rows=(300, 1, 4000, 77, 9), pool=6):
    rng = np.random.default_rng(seed)
    rows = np.array(rows[:T], np.int64)
    off = np.zeros(T + 1, np.int64)
    np.cumsum(rows, out=off[1:])
    lengths = rng.integers(0, 2 * pool + 1, size=T * B)
    bo = np.zeros(T * B + 1, np.int64)
    np.cumsum(lengths, out=bo[1:])
    t_of_bag = np.repeat(np.arange(T), B)
    t_of_pair = np.repeat(t_of_bag, lengths)
    idx = (rng.random(len(t_of_pair)) * rows[t_of_pair]).astype(np.int32)
    return off, bo.astype(np.int32), idx, T, B, int(off[-1])


def check(off, bo, idx, T, B, total_rows, bound=0, want=None):
    ref = expected(off, bo, idx, T, B, total_rows, bound)
    if want is not None:
        assert ref == want, (ref, want)   # the planted problem is what the definition finds
    got = run(off, bo, idx, T, B, total_rows, bound)
    assert got == ref, (got, ref)
    return got


def test_valid_workloads():
    for cfg in ("c1", "c2"):
        w = wl.WORKLOADS[cfg]
        b = wl.make_batch(w, 0)
        print(f"\n[{cfg}] pairs {b.num_pairs}", flush=True)
        for bound in (w.rows_per_table, 0):
            assert check(b.table_row_offset, b.bag_offsets, b.indices, w.num_tables, w.batch,
                         w.total_rows, bound) == OK


def test_planted_index_errors():
    off, bo, idx, T, B, R = layout(1)
    n = len(idx)
    j0, j1 = n // 3, 2 * n // 3
    # the table of pair j1 and its row count
    t1 = int(np.searchsorted(bo[np.arange(T) * B], j1, side="right") - 1)
    a = idx.copy(); a[j1] = off[t1 + 1] - off[t1]               # one past its table
    check(off, bo, a, T, B, R, want=(tc.TC_INDEX_OUT_OF_RANGE, j1))
    a[j0] = -1                                                   # a lower one wins
    check(off, bo, a, T, B, R, want=(tc.TC_INDEX_OUT_OF_RANGE, j0))
    a = idx.copy(); a[n - 1] = 2 ** 31 - 1                        # the last pair
    check(off, bo, a, T, B, R, want=(tc.TC_INDEX_OUT_OF_RANGE, n - 1))
    a = idx.copy(); a[0] = -2 ** 31                               # the first pair
    check(off, bo, a, T, B, R, want=(tc.TC_INDEX_OUT_OF_RANGE, 0))


def test_bound_on_table_rows():
    # indices inside their tables but at or above the caller's bound
    off, bo, idx, T, B, R = layout(2)
    big = int(np.argmax(off[1:] - off[:-1]))            # the 4000-row table
    pairs = np.arange(bo[big * B], bo[(big + 1) * B])
    j = int(pairs[len(pairs) // 2])
    a = idx.copy(); a[j] = 3999
    assert check(off, bo, a, T, B, R, bound=0) == OK
    assert check(off, bo, a, T, B, R, bound=4000) == OK
    check(off, bo, a, T, B, R, bound=3999, want=(tc.TC_INDEX_OUT_OF_RANGE, j))


def test_planted_offset_errors():
    off, bo, idx, T, B, R = layout(3)
    TB = T * B
    b = bo.copy(); b[0] = 1
    check(off, b, idx, T, B, R, want=(tc.TC_INDEX_BAD_BAG_OFFSETS, 0))
    b = bo.copy(); b[TB] = len(idx) - 1
    check(off, b, idx, T, B, R, want=(tc.TC_INDEX_BAD_BAG_OFFSETS, TB))
    b = bo.copy(); b[17] = b[16] - 1
    check(off, b, idx, T, B, R, want=(tc.TC_INDEX_BAD_BAG_OFFSETS, 17))
    b = bo.copy(); b[9] = 2 ** 31 - 1                               # far past the pairs
    check(off, b, idx, T, B, R, want=(tc.TC_INDEX_BAD_BAG_OFFSETS, 10))
    o = off.copy(); o[0] = 5
    check(o, bo, idx, T, B, R, want=(tc.TC_INDEX_BAD_TABLE_OFFSETS, 0))
    o = off.copy(); o[T] = R + 1
    check(o, bo, idx, T, B, R, want=(tc.TC_INDEX_BAD_TABLE_OFFSETS, T))
    o = off.copy(); o[2] = o[1] - 1
    check(o, bo, idx, T, B, R, want=(tc.TC_INDEX_BAD_TABLE_OFFSETS, 2))
    # the lowest kind wins over lower positions of later kinds
    a = idx.copy(); a[0] = -1
    b = bo.copy(); b[TB] = len(idx) + 1
    check(off, b, a, T, B, R, want=(tc.TC_INDEX_BAD_BAG_OFFSETS, TB))
    o = off.copy(); o[T] = R - 1
    check(o, b, a, T, B, R, want=(tc.TC_INDEX_BAD_TABLE_OFFSETS, T))


def test_empty_and_degenerate_layouts():
    z = np.zeros(0, np.int32)
    assert check(np.array([0], np.int64), np.array([0], np.int32), z, 0, 0, 0) == OK
    assert check(np.array([0, 10], np.int64), np.zeros(5, np.int32), z, 1, 4, 10) == OK
    # pairs but no bags: the bag offsets cannot account for them
    check(np.array([0, 10], np.int64), np.array([0], np.int32), np.zeros(3, np.int32), 1, 0, 10,
          want=(tc.TC_INDEX_BAD_BAG_OFFSETS, 0))
    # a table without rows cannot hold a pair
    check(np.array([0, 0, 5], np.int64), np.array([0, 1, 2], np.int32),
          np.array([0, 4], np.int32), 2, 1, 5, want=(tc.TC_INDEX_OUT_OF_RANGE, 0))
    # tables without pairs are passed over
    assert check(np.array([0, 3, 6, 9], np.int64), np.array([0, 0, 2, 2], np.int32),
                 np.array([2, 1], np.int32), 3, 1, 9) == OK


def test_many_tables_and_stale_report():
    # more tables than are staged in LDS: the table search runs in memory
    T, B = 1500, 2
    off, bo, idx, T, B, R = layout(4, T=T, B=B, rows=tuple([7, 1, 30] * 500), pool=2)
    assert check(off, bo, idx, T, B, R) == OK
    j = len(idx) - 5
    t = int(np.searchsorted(bo[np.arange(T) * B], j, side="right") - 1)
    a = idx.copy(); a[j] = off[t + 1] - off[t]
    report = torch.full((2,), 123, dtype=torch.int64, device=DEV)
    assert run(off, bo, a, T, B, R, 0, report) == (tc.TC_INDEX_OUT_OF_RANGE, j)
    # the same report buffer again: the old result does not leak into the new one
    assert run(off, bo, idx, T, B, R, 0, report) == OK


def test_random_corruptions():
    rng = np.random.default_rng(11)
    for trial in range(12):
        off, bo, idx, T, B, R = layout(100 + trial)
        off, bo, idx = off.copy(), bo.copy(), idx.copy()
        for _ in range(int(rng.integers(1, 4))):
            what = rng.integers(0, 6)
            if what == 0 and len(idx):
                idx[rng.integers(0, len(idx))] = rng.integers(-5, 5000)
            elif what == 1:
                bo[rng.integers(0, len(bo))] += int(rng.integers(-3, 4))
            elif what == 2:
                off[rng.integers(0, len(off))] += int(rng.integers(-2, 3))
            elif len(idx):
                idx[rng.integers(0, len(idx))] = -1 - rng.integers(0, 3)
        check(off, bo, idx, T, B, R, bound=int(rng.choice([0, 300, 4000])))


def test_full_size_uniform_batch():
    """32 tables x 1M rows, 5.2M pairs: one bad index near the end is found."""
    w = wl.WORKLOADS["c4"]
    b = wl.make_batch(w, 0)
    n = b.num_pairs
    print(f"\n[c4] pairs {n}", flush=True)
    assert run(b.table_row_offset, b.bag_offsets, b.indices, w.num_tables, w.batch,
               w.total_rows, w.rows_per_table) == OK
    a = b.indices.copy()
    j = n - 1000
    a[j] = w.rows_per_table
    assert run(b.table_row_offset, b.bag_offsets, a, w.num_tables, w.batch, w.total_rows,
               0) == (tc.TC_INDEX_OUT_OF_RANGE, j)
