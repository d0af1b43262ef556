"""The multi-threaded CPU baseline (cpu_baseline/, a reported baseline of
the benchmark) equals the single-threaded fp32 oracle bit for bit: forward
rows, coalesced rows and their order, updated table and accumulator rows,
on seeded inputs of each workload's distributions (CPU only)."""
import numpy as np
import pytest

import cpu_baseline
import oracle
from paper_2010_13100_amd import workload as wl

W = wl.WORKLOADS
SHAPES = {
    "c1": W["c1"],
    "c2-2x20k": W["c2"].scaled(name="c2-2x20k", num_tables=2, rows_per_table=20_000, batch=256),
    "c3-2x50k": W["c3"].scaled(name="c3-2x50k", num_tables=2, rows_per_table=50_000, batch=256),
    "c4-4x20k": W["c4"].scaled(name="c4-4x20k", num_tables=4, rows_per_table=20_000, batch=513),
    "c5-1x200k": W["c5"].scaled(name="c5-1x200k", num_tables=1, rows_per_table=200_000,
                                batch=509),
}


@pytest.mark.parametrize("name", list(SHAPES))
def test_matches_oracle_bit_for_bit(name):
    w = SHAPES[name]
    b = wl.make_batch(w, step=0)
    orc = oracle.Oracle("f32")
    src, _ = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                b.bag_offsets)
    ids = np.unique(src)
    table0 = wl.table_rows(w, ids)
    ref = oracle.train_step(orc, num_tables=w.num_tables, bags_per_table=w.batch,
                            table_row_offset=b.table_row_offset, indices=b.indices,
                            bag_offsets=b.bag_offsets, grad_out=b.grad_out, table=table0,
                            table_ids=ids, optimizer=w.optimizer, lr=np.float32(w.lr),
                            eps=np.float32(w.eps))
    cb = cpu_baseline.CpuBaseline()
    table = table0.copy()
    acc = np.zeros_like(table) if w.optimizer == "adagrad" else None
    out, coal, rows, _ = cb.train_step(b.bag_offsets, np.searchsorted(ids, src), table,
                                       b.grad_out, w.optimizer, acc, np.float32(w.lr),
                                       np.float32(w.eps))
    assert np.array_equal(out, ref.out)
    assert np.array_equal(ids[rows], ref.coal_rows)
    assert np.array_equal(coal, ref.coal)
    assert np.array_equal(table, ref.table)
    if acc is not None:
        assert np.array_equal(acc, ref.acc)
    assert cb.threads >= 1


def test_empty_bags_and_no_pairs():
    cb = cpu_baseline.CpuBaseline()
    table = np.ones((3, 8), np.float32)
    out, coal, rows, _ = cb.train_step(np.zeros(4, np.int32), np.zeros(0, np.int32), table,
                                       np.ones((3, 8), np.float32))
    assert not out.any() and len(coal) == 0 and len(rows) == 0
    assert (table == 1).all()
