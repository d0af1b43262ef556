"""Edge cases of the HIP path against the CPU oracle: empty bags and empty
batches, a single pair, every pair on one row, all rows distinct, the last
row id, segments longer than a sort tile, and every lane shape of dim."""
import numpy as np
import pytest

from paper_2010_13100_amd import workload as wl
from tests.gpu_harness import DeviceRun, OracleModel, assert_close, compare_cast

pytestmark = pytest.mark.gpu


def custom(num_tables, rows, dim, bags, seed=0, optimizer="sgd"):
    """Workload + batch from explicit bag lists (bags[t][b] = table-local rows)."""
    batch = len(bags[0])
    assert all(len(bt) == batch for bt in bags)
    w = wl.Workload(f"edge-{num_tables}x{rows}-d{dim}", 900 + seed, num_tables, rows, dim, batch,
                    "fixed", 1, "uniform", optimizer=optimizer)
    lengths = [len(bag) for bt in bags for bag in bt]
    off = np.zeros(len(lengths) + 1, np.int64)
    np.cumsum(lengths, out=off[1:])
    flat = [r for bt in bags for bag in bt for r in bag]
    rng = np.random.default_rng(seed)
    b = wl.Batch(np.asarray(flat, np.int32).reshape(-1), off.astype(np.int32),
                 wl.table_row_offsets(w),
                 rng.standard_normal((w.num_bags, dim), dtype=np.float32))
    return w, b


def check(w, b):
    """Both step forms (backward + update as two calls and fused) against the
    oracle; returns the cast of the fused run."""
    for fused in (False, True):
        cast = check_one(w, b, fused)
    return cast


def check_one(w, b, fused):
    print(f"\n[{w.name} fused={fused}] pairs {b.num_pairs}", flush=True)
    run = DeviceRun(w, max_pairs=max(b.num_pairs, 1))
    t = np.repeat(np.arange(w.num_bags) // w.batch, np.diff(b.bag_offsets))
    touched = np.unique(b.table_row_offset[t] + b.indices)
    model = OracleModel(w, touched if len(touched) else np.zeros(1, np.int64))
    out, cast, coal = run.step(b, fused=fused)
    r_out, r_cast, r_coal, _ = model.step(b)
    assert_close(out, r_out, "forward out", bitwise=True)
    compare_cast(cast, r_cast, b.num_pairs)
    assert_close(coal, r_coal, "coalesced gradient", bitwise=True)
    if len(touched):
        assert_close(run.rows(touched), model.rows(touched), "table rows", bitwise=True)
        if w.optimizer == "adagrad":
            assert_close(run.acc_rows(touched), model.acc[np.searchsorted(model.ids, touched)],
                         "accumulator", bitwise=True)
    run.release()
    return cast


def test_empty_batch():
    w, b = custom(2, 50, 8, [[[], [], []], [[], [], []]])
    cast = check(w, b)
    assert cast["num_unique"] == 0 and cast["seg_offsets"].tolist() == [0]


def test_empty_bags_and_single_pair():
    w, b = custom(1, 10, 16, [[[], [9], []]])
    cast = check(w, b)
    assert cast["unique_rows"].tolist() == [9]


def test_paper_worked_example():
    w, b = custom(1, 5, 4, [[[1, 2, 4], [0, 2]]])
    cast = check(w, b)
    assert cast["casted_src"].tolist() == [1, 0, 0, 1, 0]
    assert cast["casted_dst"].tolist() == [0, 1, 2, 2, 3]
    assert cast["unique_rows"].tolist() == [0, 1, 2, 4]
    assert cast["seg_offsets"].tolist() == [0, 1, 2, 4, 5]


def test_all_pairs_on_one_row():
    # one segment of 9000 pairs: longer than two sort tiles
    bags = [[[7] * 30 for _ in range(300)]]
    w, b = custom(1, 100, 64, bags)
    cast = check(w, b)
    assert cast["num_unique"] == 1 and cast["seg_offsets"].tolist() == [0, 9000]


def test_all_rows_distinct_and_last_row():
    rng = np.random.default_rng(1)
    perm = rng.permutation(12_000)
    last = int(np.flatnonzero(perm == 11_999)[0])
    perm[[0, last]] = perm[[last, 0]]          # the last row id comes first
    bags = [[perm[i:i + 40].tolist() for i in range(0, 12_000, 40)]]
    w, b = custom(1, 12_000, 32, bags, optimizer="adagrad")
    cast = check(w, b)
    assert cast["num_unique"] == 12_000 and cast["unique_rows"][-1] == 11_999


def test_long_segment_among_random_rows():
    rng = np.random.default_rng(2)
    bags = []
    for t in range(3):
        tb = []
        for _ in range(400):
            bag = rng.integers(0, 4000, size=60).tolist()
            bag[::2] = [4321] * 30            # row 4321 takes half of every bag
            tb.append(bag)
        bags.append(tb)
    w, b = custom(3, 5000, 128, bags, seed=2, optimizer="adagrad")
    cast = check(w, b)
    seg = np.diff(cast["seg_offsets"])
    assert seg.max() == 12_000


@pytest.mark.parametrize("dim", [4, 12, 20, 64, 128, 256, 320, 512, 1024])
def test_dims(dim):
    rng = np.random.default_rng(dim)
    bags = [[rng.integers(0, 300, size=int(rng.integers(0, 25))).tolist() for _ in range(97)]
            for _ in range(2)]
    w, b = custom(2, 300, dim, bags, seed=dim % 7, optimizer="adagrad" if dim % 3 else "sgd")
    check(w, b)
