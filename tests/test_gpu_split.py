"""The backward with its workspace: segments of at least 2048 pairs summed in
pieces (include/tc.h documents the order), against the CPU oracle.

Two references. Expected coalesced rows of split segments are composed
from the fp32 oracle's own sums in the documented order (each piece by
Algorithm 3 from +0, the piece sums added in order), so coalesced rows,
updated table rows and accumulators are compared bit for bit with the fp32
oracle run in that order. The tolerance is judged against the definition
in fp64: every coalesced row (split or not) against the fp64 sums, every
accumulator row against the fp64 pipeline (sums, then the optimizer steps),
and every table row against the fp64 optimizer steps taken at the GPU's
coalesced rows (and, for SGD, against the fp64 pipeline), all within 1e-5
row-normwise. (A chain of tens of thousands of fp32 adds can itself miss
1e-5 against the fp64 sum, which is why hot rows are split.)"""
import numpy as np
import pytest
import torch

import oracle
from paper_2010_13100_amd import tc
from paper_2010_13100_amd import workload as wl
from tests.gpu_harness import (DeviceRun, OracleModel, assert_close, check_against_definition,
                               check_step_against_definition, compare_cast, is_split, to_dev)

pytestmark = pytest.mark.gpu

W = wl.WORKLOADS
# Zipf shapes whose hottest rows reach past 2048 pairs
SHAPES = {
    "c2-2x20k": W["c2"].scaled(name="c2-2x20k", num_tables=2, rows_per_table=20_000, batch=256),
    "c5-1x200k": W["c5"].scaled(name="c5-1x200k", num_tables=1, rows_per_table=200_000, batch=509),
    "c3-2x50k-b1024": W["c3"].scaled(name="c3-2x50k-b1024", num_tables=2, rows_per_table=50_000,
                                     batch=1024),
}


def global_rows(w, b):
    t = np.repeat(np.arange(w.num_bags) // w.batch, np.diff(b.bag_offsets))
    return b.table_row_offset[t] + b.indices


def run_steps(w, batches, fused, run=None, cap=None):
    touched = np.unique(np.concatenate([global_rows(w, b) for b in batches]))
    if run is None:
        run = DeviceRun(w, max_pairs=max(b.num_pairs for b in batches), split_long=True)
    model = OracleModel(w, touched, split_cap=run.split_cap if cap is None else cap)
    model64 = OracleModel(w, touched, precision="f64")
    shadow64 = OracleModel(w, touched, precision="f64")
    nsplit = 0
    chains = []
    for b in batches:
        out, cast, coal = run.step(b, fused=fused)
        r_out, r_cast, r_coal, r_rows = model.step(b)
        _, _, coal64, _ = model64.step(b)
        out64, _, _, _ = shadow64.step(b, coal_override=coal)
        chains.append(check_step_against_definition(cast, model.split, out, out64, coal,
                                                    coal64, w.name))
        assert_close(out, r_out, "forward out", bitwise=True)
        compare_cast(cast, r_cast, b.num_pairs)
        assert_close(coal, r_coal, "coalesced gradient (pieces)", bitwise=True)
        nsplit += len(model.split)
    assert_close(run.rows(touched), model.table, "updated table rows", bitwise=True)
    if model.acc is not None:
        acc = run.acc_rows(touched)
        assert_close(acc.reshape(len(touched), -1), model.acc.reshape(len(touched), -1),
                     "accumulator", bitwise=True)
    # every touched row (split or one chain) after the steps, against the
    # fp64 definition: sums and optimizer steps in double
    check_against_definition(run, model64, shadow64, w.name, np.concatenate(chains))
    print(f"split segments over the steps: {nsplit}", flush=True)
    return run, nsplit


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("name", list(SHAPES))
def test_split_steps_match_oracle(name, fused):
    w = SHAPES[name]
    batches = [wl.make_batch(w, s) for s in (0, 1)]
    print(f"\n[{name} fused={fused}] pairs {[b.num_pairs for b in batches]}", flush=True)
    run, nsplit = run_steps(w, batches, fused)
    assert nsplit > 0
    run.release()


def hot_batch(lengths, dim, rows=1000, filler=20_000, bag=64, seed=0, optimizer="adagrad",
              hot_rows=None):
    """One table: row hot_rows[k] gathered lengths[k] times, plus `filler`
    uniform pairs over the other rows, shuffled into bags of `bag` pairs."""
    rng = np.random.default_rng(seed)
    hot = (np.asarray(hot_rows) if hot_rows is not None
           else rng.choice(rows, size=len(lengths), replace=False))
    pool = np.setdiff1d(np.arange(rows), hot)
    flat = np.concatenate([np.repeat(hot, lengths), rng.choice(pool, size=filler)])
    rng.shuffle(flat)
    nb = (len(flat) + bag - 1) // bag
    off = np.minimum(np.arange(nb + 1) * bag, len(flat))
    w = wl.Workload(f"hot-d{dim}", 970 + seed, 1, rows, dim, nb, "fixed", bag, "uniform",
                    optimizer=optimizer)
    b = wl.Batch(flat.astype(np.int32), off.astype(np.int32), wl.table_row_offsets(w),
                 rng.standard_normal((nb, dim), dtype=np.float32))
    return w, b


@pytest.mark.parametrize("dim", [4, 64, 260, 1024])
def test_piece_counts_at_their_edges(dim):
    # split or not (2047 / 2048), n = 2 / 3 pieces (3071 / 3072), n = 32
    # exactly (32768) and capped (33792, 70001)
    lengths = [2047, 2048, 2049, 3071, 3072, 32768, 33792, 70001]
    if dim == 1024:
        lengths = [2047, 2048, 3072, 33792]
    w, b = hot_batch(lengths, dim, seed=dim)
    for fused in (True, False):
        print(f"\n[d{dim} fused={fused}] pairs {b.num_pairs}", flush=True)
        run, nsplit = run_steps(w, [b], fused)
        assert nsplit == len(lengths) - 1
        run.release()


def test_rmsprop_pieces():
    w, b = hot_batch([5000, 40000], 128, seed=5, optimizer="rmsprop")
    run, nsplit = run_steps(w, [b], True)
    assert nsplit == 2
    run.release()


def test_stale_and_garbage_workspace():
    """A workspace of random contents, then reused by a second batch whose
    split segments sit elsewhere: entries of other calls are never taken."""
    w = SHAPES["c2-2x20k"]
    b0, b1 = wl.make_batch(w, 0), wl.make_batch(w, 5)
    run = DeviceRun(w, max_pairs=max(b0.num_pairs, b1.num_pairs), split_long=True)
    ws = run.trainer.bwd_workspace
    gen = torch.Generator(device="cuda").manual_seed(3)
    ws.view(torch.int32)[:] = torch.randint(-5, 2000, (ws.numel() // 4,), generator=gen,
                                            device="cuda", dtype=torch.int32)
    run_steps(w, [b0, b1], True, run=run)
    run.release()


def test_workspace_covering_part_of_the_batch():
    """Sized for half the pairs: the early hot row (low row id, so early in
    sorted order) is split, the late one is summed as one chain."""
    w, b = hot_batch([9000, 9000], 64, rows=1000, filler=22_000, seed=7, hot_rows=[3, 996])
    half = b.num_pairs // 2
    run = DeviceRun(w, max_pairs=b.num_pairs, split_long=True)
    small = tc.tc_backward_workspace_bytes(half, w.dim)
    run.trainer.bwd_workspace = torch.empty(small, dtype=torch.uint8, device="cuda")
    # the cover is at least `half` pairs and, from the layout, less than
    # half + 8192: the late row's segment starts past that either way
    so = np.concatenate([[0], np.cumsum(np.bincount(b.indices, minlength=w.rows_per_table))])
    assert so[3] + 9000 <= half and so[996] > half + 8192
    _, nsplit = run_steps(w, [b], True, run=run, cap=half)
    assert nsplit == 1
    run.release()


def test_no_workspace_is_one_chain():
    w, b = hot_batch([9000], 64, seed=9)
    run = DeviceRun(w, max_pairs=b.num_pairs, split_long=False)
    assert run.trainer.bwd_workspace is None
    _, nsplit = run_steps(w, [b], True, run=run)
    assert nsplit == 0
    run.release()


def test_repeats_bit_for_bit():
    w = SHAPES["c5-1x200k"]
    b = wl.make_batch(w, 2)
    res = []
    for _ in range(2):
        run = DeviceRun(w, max_pairs=b.num_pairs, split_long=True)
        out, cast, coal = run.step(b, fused=True)
        res.append((coal, run.trainer.W.cpu().numpy()))
        run.release()
    assert np.array_equal(res[0][0], res[1][0]) and np.array_equal(res[0][1], res[1][1])


def test_baseline_coalesce_pieces_equal_casted():
    w = SHAPES["c2-2x20k"]
    b = wl.make_batch(w, 0)
    run = DeviceRun(w, max_pairs=b.num_pairs, split_long=True)
    t = run.trainer
    off, idx, bo, g = (to_dev(b.table_row_offset), to_dev(b.indices), to_dev(b.bag_offsets),
                       to_dev(b.grad_out))
    t.cast(off, idx, bo, b.num_pairs)
    t.backward(g)
    torch.cuda.synchronize()
    u = int(t.num_unique.item())
    casted = t.coal[:u].cpu().numpy()
    t.baseline_backward(off, idx, bo, b.num_pairs, g)
    torch.cuda.synchronize()
    assert np.array_equal(t.coal[:u].cpu().numpy(), casted)
    so = t.seg_offsets[:u + 1].cpu().numpy()
    assert any(is_split(so[k], so[k + 1] - so[k], run.split_cap) for k in range(u))
    run.release()
