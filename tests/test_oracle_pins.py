"""The CPU oracle against the paper's worked example, closed forms,
invariants, brute force and a-priori rounding-error bounds (no GPU)."""
import numpy as np
import pytest

import oracle
from paper_2010_13100_amd import workload as wl
from tests import pins


@pytest.fixture(scope="module", params=["f64", "f32"])
def orc(request):
    return oracle.Oracle(request.param)


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)


@pytest.fixture(scope="module")
def both():
    return oracle.Oracle("f32"), oracle.Oracle("f64")


@pytest.mark.parametrize("cfg", ["c1", "c2", "c3", "c4", "c5"])
def test_f32_within_rounding_bound_of_f64(both, cfg):
    """The fp32 oracle stays within the a-priori rounding bound of the fp64
    oracle on small instances with each workload's distributions."""
    w = wl.WORKLOADS[cfg]
    small = w.scaled(name=cfg + "-tiny", num_tables=min(w.num_tables, 3),
                     rows_per_table=min(w.rows_per_table, 5000), batch=64)
    b = wl.make_batch(small, step=1)
    pins.check_f32_against_f64(*both, small, b)


def test_train_step_equivalences(both):
    """train_step: Algorithm 1 (baseline backward) and Algorithm 3 give the same
    coalesced gradients; untouched rows of the table keep their values."""
    orc32, _ = both
    w = wl.WORKLOADS["c3"].scaled(name="c3-tiny", num_tables=2, rows_per_table=3000, batch=128)
    b = wl.make_batch(w, step=0)
    tbl = wl.table_rows(w, np.arange(w.total_rows))
    res = oracle.train_step(orc32, num_tables=w.num_tables, bags_per_table=w.batch,
                            table_row_offset=b.table_row_offset, indices=b.indices,
                            bag_offsets=b.bag_offsets, grad_out=b.grad_out, table=tbl,
                            optimizer="adagrad", lr=w.lr, eps=w.eps)
    c = res.cast
    coal3 = orc32.casted_gather_reduce(c["casted_src"], c["casted_dst"], b.grad_out, c["num_unique"])
    assert np.array_equal(coal3, res.coal)
    assert np.array_equal(res.coal_rows, c["unique_rows"])
    untouched = np.setdiff1d(np.arange(w.total_rows), c["unique_rows"])
    assert np.array_equal(res.table[untouched], tbl[untouched])
    assert np.all(res.acc[untouched] == 0)
    assert np.all(res.table[c["unique_rows"]] != tbl[c["unique_rows"]])
