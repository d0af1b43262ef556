"""The paper's baseline backward on the GPU (gradient expand, stable argsort,
Algorithm 1's accumulate) against the CPU oracle, and against the casted
backward of the same batch: Algorithm 1 and Algorithm 3 give the same
coalesced gradients, row for row and bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from paper_2010_13100_amd import workload as wl
from tests.gpu_harness import DeviceRun, assert_close, to_dev
from tests.test_gpu_parity import SMALL

pytestmark = pytest.mark.gpu


def run_both(w, b):
    """Casted backward, then the baseline on the same trainer; returns both
    results and the oracle's."""
    run = DeviceRun(w, max_pairs=max(b.num_pairs, 1))
    t = run.trainer
    off, idx, bo, g = (to_dev(b.table_row_offset), to_dev(b.indices), to_dev(b.bag_offsets),
                       to_dev(b.grad_out))
    t.cast(off, idx, bo, b.num_pairs)
    t.backward(g)
    torch.cuda.synchronize()
    u = int(t.num_unique.item())
    casted = dict(unique_rows=t.unique_rows[:u].cpu().numpy(),
                  seg_offsets=t.seg_offsets[:u + 1].cpu().numpy(),
                  coal=t.coal[:u].cpu().numpy())
    t.baseline_backward(off, idx, bo, b.num_pairs, g)
    torch.cuda.synchronize()
    u2 = int(t.num_unique.item())
    base = dict(unique_rows=t.unique_rows[:u2].cpu().numpy(),
                seg_offsets=t.seg_offsets[:u2 + 1].cpu().numpy(),
                sorted_pos=t.casted_src[:b.num_pairs].cpu().numpy(),
                expanded=t.expanded[:b.num_pairs].cpu().numpy(),
                coal=t.coal[:u2].cpu().numpy())
    run.release()
    orc = oracle.Oracle("f32")
    src, dst = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                  b.bag_offsets)
    exp = orc.expand(dst, b.grad_out)
    coal, rows = orc.coalesce(src, exp)
    ref = dict(src=src, expanded=exp, coal=coal, rows=rows)
    return casted, base, ref


@pytest.mark.parametrize("name", list(SMALL))
def test_baseline_matches_oracle_and_casted(name):
    w = SMALL[name]
    b = wl.make_batch(w, 0)
    print(f"\n[{name}] pairs {b.num_pairs}", flush=True)
    casted, base, ref = run_both(w, b)
    assert np.array_equal(base["expanded"], ref["expanded"])
    assert np.array_equal(base["sorted_pos"], np.argsort(ref["src"], kind="stable"))
    assert np.array_equal(base["unique_rows"], ref["rows"])
    assert_close(base["coal"], ref["coal"], "baseline coalesced gradient", bitwise=True)
    # Algorithm 1 (expand-coalesce) = Algorithm 3 (casted gather-reduce)
    assert np.array_equal(base["unique_rows"], casted["unique_rows"])
    assert np.array_equal(base["seg_offsets"], casted["seg_offsets"])
    assert np.array_equal(base["coal"], casted["coal"])


def test_baseline_long_segment_and_empty_bags():
    # 9000 pairs on one row (the long-segment path) plus empty bags
    bags = [[[7] * 30 if k % 3 else [] for k in range(450)]]
    w = wl.Workload("baseline-long", 950, 1, 100, 64, len(bags[0]), "fixed", 1, "uniform")
    lengths = [len(x) for x in bags[0]]
    off = np.zeros(len(lengths) + 1, np.int64)
    np.cumsum(lengths, out=off[1:])
    rng = np.random.default_rng(3)
    b = wl.Batch(np.asarray([r for x in bags[0] for r in x], np.int32), off.astype(np.int32),
                 wl.table_row_offsets(w), rng.standard_normal((w.num_bags, 64), dtype=np.float32))
    casted, base, ref = run_both(w, b)
    assert base["seg_offsets"].tolist() == [0, 9000]
    assert_close(base["coal"], ref["coal"], "baseline coalesced gradient", bitwise=True)
    assert np.array_equal(base["coal"], casted["coal"])
