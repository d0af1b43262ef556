"""All five workloads at full size, one step each, in the launch
configuration the benchmark times (forward and cast as one call, backward
and update as one, with the backward workspace, so segments of 2048 pairs
or more are summed in pieces; the coalesced rows are also stored, to be
checked, except in the cases that pass exactly the benchmark's arguments).
The casted index is
compared with the oracle's in full (bit for bit); forward rows, coalesced
gradients and updated rows are compared on samples the oracle computes on
their own: a sampled bag needs only its own pairs, a sampled table row only
the pairs that gather it (kept in input order, so the sum order is
unchanged). A split row's expected sum is composed from the oracle's sums
in the documented piece order (bit for bit), and the sampled rows' updated
table and accumulator values are also checked against the fp64 definition
(fp64 sums, then the optimizer step in double) within the tolerance."""
import numpy as np
import pytest
import torch

import oracle
from paper_2010_13100_amd import workload as wl
from tests.gpu_harness import (FP32_CHAIN_LIMIT, SPLIT_PAIRS, DeviceRun, assert_close,
                               check_step_slope, compare_cast, piecewise_row, scatter, step_slope)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg,split,opt,stored", [
    ("c1", True, None, True), ("c2", True, None, True), ("c3", True, None, True),
    ("c4", True, None, True), ("c5", True, None, True), ("c2", False, None, True),
    ("c3", False, None, True), ("c3", True, "rmsprop", True), ("c2", True, None, False),
    ("c5", True, None, False)])
def test_full_size_step(cfg, split, opt, stored):
    """split: with the backward workspace (as the benchmark runs), or without
    it (every segment one ordered chain, the hottest rows included). opt:
    another optimizer than the workload's (the same batch and table).
    stored: casted_dst and the coalesced rows written too; without them the
    calls take exactly the benchmark's arguments, and the coalesced rows are
    checked through the updated table rows only."""
    w = wl.variant(wl.WORKLOADS[cfg], optimizer=opt)
    b = wl.make_batch(w, step=0)
    print(f"\n[{cfg} split={split} stored={stored}] {w.name}: {b.num_pairs} pairs", flush=True)
    run = DeviceRun(w, max_pairs=b.num_pairs, split_long=split)
    assert run.split_cap >= b.num_pairs if split else run.split_cap == 0
    run.run_step(b, with_casted_dst=stored, fused=True, store_coal=stored)
    t = run.trainer
    orc = oracle.Oracle("f32")
    src, dst = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                  b.bag_offsets)
    ref_cast = orc.tensor_casting(src, dst)
    got_cast = run.fetch_cast()
    compare_cast(got_cast, ref_cast, b.num_pairs)
    print(f"[{cfg}] cast bit-exact: U = {got_cast['num_unique']}", flush=True)
    rng = np.random.default_rng(1)

    # forward: 256 sampled bags
    bags = np.sort(rng.choice(w.num_bags, size=min(256, w.num_bags), replace=False))
    lo, hi = b.bag_offsets[bags], b.bag_offsets[bags + 1]
    sel = np.concatenate([np.arange(a, c) for a, c in zip(lo, hi)])
    s_src = src[sel]
    s_dst = np.repeat(np.arange(len(bags)), hi - lo).astype(np.int32)
    ids = np.unique(s_src)
    ref_out = orc.forward(s_src, s_dst, len(bags), wl.table_rows(w, ids), ids)
    got_out = t.out.index_select(0, torch.from_numpy(bags).cuda()).cpu().numpy()
    assert_close(got_out, ref_out, f"{cfg} forward (sampled bags)", bitwise=True)

    # backward + update: the 16 longest segments and 1000 random rows
    seg = np.diff(ref_cast["seg_offsets"])
    uniq = ref_cast["unique_rows"]
    pick = np.unique(np.concatenate([np.argsort(seg)[-16:],
                                     rng.choice(len(uniq), size=min(1000, len(uniq)),
                                                replace=False)]))
    rows = uniq[pick]
    mask = np.isin(src, rows)
    ref_coal, ref_rows = orc.coalesce(src[mask], orc.expand(dst[mask], b.grad_out))
    assert np.array_equal(ref_rows, rows)
    orc64 = oracle.Oracle("f64")
    seq64, _ = orc64.coalesce(src[mask], orc64.expand(dst[mask], b.grad_out))
    pieces = np.flatnonzero(seg[pick] >= SPLIT_PAIRS) if run.split_cap else np.zeros(0, int)
    for k in pieces:   # the row's bags in input order = its segment in sorted order
        ref_coal[k] = piecewise_row(orc, dst[src == rows[k]], b.grad_out)
    if stored:
        got_coal = t.coal.index_select(0, torch.from_numpy(pick).cuda()).cpu().numpy()
        assert_close(got_coal, ref_coal, f"{cfg} coalesced gradient (sampled rows)",
                     bitwise=True)
    tbl = wl.table_rows(w, rows)
    acc = None if w.optimizer == "sgd" else np.zeros_like(tbl)
    scatter(orc, w, rows, ref_coal, tbl, acc, rows)
    got_w = run.rows(rows)
    got_a = None if acc is None else run.acc_rows(rows)
    if acc is not None:
        assert_close(got_a, acc, f"{cfg} accumulator (sampled rows)", bitwise=True)
    assert_close(got_w, tbl, f"{cfg} updated rows (sampled)", bitwise=True)
    # the same rows against the definition in fp64. Rows the benchmark's
    # configuration sums (split rows and chains under 2048 pairs) must be
    # within the tolerance; without the workspace, chains longer than
    # FP32_CHAIN_LIMIT are the literal sequential fp32 sum, checked bit for
    # bit above only. The step from A = 0 is checked three ways: accumulator
    # rows against the fp64 pipeline; table rows against the fp64 step
    # taken at the GPU's coalesced rows (when they are stored; they are
    # checked against the fp64 sums above); and table rows against the fp64
    # pipeline within the tolerance on G carried through the step's slope
    # (and, for SGD, whose step is linear, within the tolerance itself).
    near = np.flatnonzero((seg[pick] < FP32_CHAIN_LIMIT) | (seg[pick] >= SPLIT_PAIRS)
                          if run.split_cap else seg[pick] < FP32_CHAIN_LIMIT)
    if run.split_cap:
        assert len(near) == len(rows)
    tbl64 = wl.table_rows(w, rows).astype(np.float64)
    acc64 = None if acc is None else np.zeros_like(tbl64)
    scatter(orc64, w, rows, seq64, tbl64, acc64, rows)
    if acc is not None:
        assert_close(got_a[near], acc64[near], f"{cfg} accumulator vs fp64 definition")
    check_step_slope(got_w[near], tbl64[near], step_slope(w, seq64[near]), seq64[near],
                     f"{cfg} updated rows vs fp64 definition")
    if w.optimizer == "sgd":
        assert_close(got_w[near], tbl64[near], f"{cfg} updated rows vs fp64 definition")
    if stored:
        assert_close(got_coal[near], seq64[near], f"{cfg} coalesced rows vs fp64 sums")
        at_g = wl.table_rows(w, rows).astype(np.float64)
        acc_g = None if acc is None else np.zeros_like(at_g)
        scatter(orc64, w, rows, got_coal.astype(np.float64), at_g, acc_g, rows)
        assert_close(got_w, at_g, f"{cfg} updated rows vs fp64 step at the GPU's G")
    print(f"[{cfg}] longest segment {seg.max()}, sampled rows {len(rows)} match "
          f"({len(pieces)} split)", flush=True)

    # rows the step does not touch keep their initial values
    cand = rng.integers(0, w.total_rows, size=5000)
    untouched = np.setdiff1d(cand, uniq)
    assert np.array_equal(run.rows(untouched), wl.table_rows(w, untouched))
    run.release()
