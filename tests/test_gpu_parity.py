"""The HIP path against the CPU oracle on the same seeded inputs.

Index outputs must match bit for bit. fp32 outputs are checked bit for
bit against the fp32 oracle (both sides add the same terms in the same
order), and within 1e-5 row-normwise relative error against the fp64
definition: forward rows and coalesced gradients against the fp64 sums,
accumulators against the fp64 pipeline, table rows against the fp64
optimizer steps taken at the GPU's coalesced rows (and, for SGD, against the
fp64 pipeline). Without a backward workspace (as here) a segment of 2048
pairs or more is one literal fp32 chain: its row is checked bit for bit
only."""
import numpy as np
import pytest
import torch

from paper_2010_13100_amd import workload as wl
from tests.gpu_harness import (DeviceRun, OracleModel, assert_close, check_against_definition,
                               check_step_against_definition, compare_cast)

pytestmark = pytest.mark.gpu

W = wl.WORKLOADS
# Each workload's distributions at sizes the oracle finishes in seconds; the
# pair counts span several 2048-pair sort tiles and end in a ragged tile.
SMALL = {
    "c1": W["c1"],
    "c2-2x20k": W["c2"].scaled(name="c2-2x20k", num_tables=2, rows_per_table=20_000, batch=256),
    "c3-2x50k": W["c3"].scaled(name="c3-2x50k", num_tables=2, rows_per_table=50_000, batch=256),
    "c4-4x20k": W["c4"].scaled(name="c4-4x20k", num_tables=4, rows_per_table=20_000, batch=513),
    "c5-1x200k": W["c5"].scaled(name="c5-1x200k", num_tables=1, rows_per_table=200_000, batch=509),
}


def global_rows(w, b):
    t = np.repeat(np.arange(w.num_bags) // w.batch, np.diff(b.bag_offsets))
    return b.table_row_offset[t] + b.indices


@pytest.mark.parametrize("bound,fused", [("table-local", True), ("table-local", False),
                                         ("global", True), ("global", False)])
@pytest.mark.parametrize("name", list(SMALL))
def test_two_steps_match_oracle(name, bound, fused):
    """bound: the cast sorts on table-local rows (the table size is passed as
    the bound) or on global rows (no bound). fused: forward and cast as one
    call (tc_embed_forward_cast) and backward and update as one
    (tc_embed_backward_update), or all four calls one by one."""
    w = SMALL[name]
    batches = [wl.make_batch(w, s) for s in (0, 1)]
    touched = np.unique(np.concatenate([global_rows(w, b) for b in batches]))
    print(f"\n[{name} {bound} fused={fused}] pairs {[b.num_pairs for b in batches]} "
          f"touched {len(touched)}", flush=True)
    run = DeviceRun(w, max_pairs=max(b.num_pairs for b in batches),
                 max_table_rows=None if bound == "table-local" else 0)
    model = OracleModel(w, touched)
    model64 = OracleModel(w, touched, precision="f64")
    shadow64 = OracleModel(w, touched, precision="f64")
    chains = []
    for b in batches:
        out, cast, coal = run.step(b, fused=fused)
        r_out, r_cast, r_coal, r_rows = model.step(b)
        _, _, coal64, _ = model64.step(b)
        out64, _, _, _ = shadow64.step(b, coal_override=coal)
        assert_close(out, r_out, "forward out", bitwise=True)
        compare_cast(cast, r_cast, b.num_pairs)
        assert np.array_equal(cast["unique_rows"], r_rows)
        assert_close(coal, r_coal, "coalesced gradient", bitwise=True)
        chains.append(check_step_against_definition(cast, [], out, out64, coal, coal64, name))
    assert_close(run.rows(touched), model.table, "updated table rows", bitwise=True)
    if w.optimizer == "adagrad":
        assert_close(run.acc_rows(touched), model.acc, "Adagrad accumulator", bitwise=True)
    check_against_definition(run, model64, shadow64, name, np.concatenate(chains))
    rng = np.random.default_rng(0)
    cand = rng.integers(0, w.total_rows, size=4000)
    untouched = np.setdiff1d(cand, touched)
    assert np.array_equal(run.rows(untouched), wl.table_rows(w, untouched))
    run.release()


def test_deterministic_across_runs():
    w = SMALL["c2-2x20k"]
    b = wl.make_batch(w, 3)
    res = []
    for _ in range(2):
        run = DeviceRun(w, max_pairs=b.num_pairs)
        out, cast, coal = run.step(b)
        res.append((out, cast["casted_src"], coal, run.trainer.W.cpu().numpy()))
        run.release()
    for a, c in zip(*res):
        assert np.array_equal(a, c)


def test_device_fill_matches_host_generator():
    from paper_2010_13100_amd import device_fill
    w = W["c5"].scaled(name="fill", rows_per_table=1000, dim=128)
    t = torch.empty((1000, 128), dtype=torch.float32, device="cuda")
    device_fill.fill_uniform(t, seed=0)
    assert np.array_equal(t.cpu().numpy(), wl.table_rows(w, np.arange(1000)))
    # rows near the end of a 50M-row table: 64-bit element counters
    first = 49_999_000
    device_fill.fill_uniform(t, seed=0, row_begin=first)
    assert np.array_equal(t.cpu().numpy(), wl.table_rows(w, np.arange(first, first + 1000)))
