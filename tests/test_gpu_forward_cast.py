"""tc_embed_forward_cast (the forward gather-reduce and Tensor Casting in one
call) against the CPU oracle: pooled rows bit for bit with the oracle's
forward (Sec. II-B), the casted index bit for bit with its Tensor Casting
(Algorithm 2). Row widths inside and outside the range whose forward runs in
the cast's own launches (dim 36..256), batches on both sides of the
single-workgroup cast (8192 pairs), table-local and global sorts, tables and
bags without pairs, and more tables than the table-local sort takes."""
import numpy as np
import pytest
import torch

import oracle
from paper_2010_13100_amd import tc
from tests.test_gpu_cast_layouts import make_case, sparse_bags_case

pytestmark = pytest.mark.gpu


def run_case(name, table_rows, pairs_per_table, bags_per_table, dim, seed, bound=None,
             case=None):
    off, bo, indices = case or make_case(table_rows, pairs_per_table, bags_per_table, seed)
    T, n, R = len(table_rows), len(indices), int(off[-1])
    bound = max(table_rows) if bound is None else bound
    print(f"\n[{name} dim={dim} bound={bound}] tables {T} pairs {n}", flush=True)
    rng = np.random.default_rng(seed + 1000)
    W = rng.standard_normal((R, dim), dtype=np.float32)
    orc = oracle.Oracle("f32")
    src, dst = orc.pairs_from_csr(T, bags_per_table, off, indices, bo)
    ref_out = orc.forward(src, dst, T * bags_per_table, W)
    ref = orc.tensor_casting(src, dst)

    dev = torch.device("cuda", 0)
    i32 = dict(dtype=torch.int32, device=dev)
    cap = max(min(n, R), 1)
    ur = torch.full((cap,), -7, **i32)
    so = torch.full((cap + 1,), -7, **i32)
    cs = torch.full((max(n, 1),), -7, **i32)
    cd = torch.full((max(n, 1),), -7, **i32)
    nu = torch.zeros(1, **i32)
    out = torch.full((T * bags_per_table, dim), float("nan"), dtype=torch.float32, device=dev)
    ws = torch.empty(max(tc.tc_cast_workspace_bytes(n, R, T), 256), dtype=torch.uint8,
                     device=dev)
    d_idx = torch.from_numpy(indices).to(dev) if n else None
    tc.tc_embed_forward_cast(torch.from_numpy(W).to(dev), torch.from_numpy(off).to(dev), T,
                             bags_per_table, bound, d_idx, torch.from_numpy(bo).to(dev), n, out,
                             ur, so, cs, cd, nu, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    same = (got == ref_out)  # the output started as NaN: every row must be written
    assert same.all(), f"forward: {np.count_nonzero(~same)} values differ"
    u = int(nu.item())
    assert u == ref["num_unique"]
    assert np.array_equal(ur[:u].cpu().numpy(), ref["unique_rows"])
    assert np.array_equal(so[:u + 1].cpu().numpy(), ref["seg_offsets"])
    assert np.array_equal(cs[:n].cpu().numpy(), ref["casted_src"][:n])
    assert np.array_equal(cd[:n].cpu().numpy(), ref["casted_dst"][:n])


@pytest.mark.parametrize("dim", [8, 36, 64, 128, 256, 260, 512])
def test_row_widths_multi_kernel(dim):
    # 14.5k pairs: the radix-sort cast; dims 36..256 run the forward in the
    # key build's launch, the others as a kernel of their own
    run_case("unequal", [5, 1000, 3, 7000, 129], [40, 3000, 7, 9000, 2500], 5, dim, seed=dim)


@pytest.mark.parametrize("dim", [8, 64, 128, 256, 512])
def test_row_widths_single_workgroup(dim):
    # 3k pairs: one cast workgroup, the forward's workgroups beside it
    run_case("small", [300, 1, 2000], [1000, 7, 2000], 11, dim, seed=dim + 1)


@pytest.mark.parametrize("n", [8191, 8192, 8193])
def test_single_workgroup_boundary(n):
    run_case(f"n={n}", [3000, 500], [n - 600, 600], 9, 64, seed=n)


def test_global_rows_and_empty_tables():
    run_case("global", [300, 400, 500, 600, 700], [0, 2500, 0, 9000, 10], 7, 128, seed=3,
             bound=0)
    run_case("empty tables", [300, 400, 500, 600, 700], [0, 2500, 0, 9000, 10], 7, 64, seed=4)


def test_many_tables():
    rng = np.random.default_rng(5)
    T = 300
    run_case("300 tables", rng.integers(1, 50, size=T).tolist(),
             rng.integers(0, 60, size=T).tolist(), 3, 64, seed=5)


def test_no_pairs():
    # every bag empty: rows of zeros and an empty casted index
    run_case("no pairs", [10, 20], [0, 0], 4, 64, seed=6)
    run_case("no pairs, narrow rows", [10, 20], [0, 0], 4, 8, seed=7)


def test_tiles_spanning_many_empty_bags():
    # pairs in every 4th bag: a sort tile spans more bags than are staged
    case = sparse_bags_case(2, 40_000, 9_000, 5000, seed=8)
    run_case("sparse bags", [5000, 5000], None, 40_000, 64, seed=8, case=case)
    case = sparse_bags_case(3, 30_000, 7_000, 5000, seed=9)
    run_case("sparse bags, global", [5000] * 3, None, 30_000, 128, seed=9, bound=0, case=case)
