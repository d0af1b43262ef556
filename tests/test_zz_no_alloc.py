"""tc_embed_backward_update_noalloc (the backward + update for callers that
cannot allocate device memory) against tc_embed_backward_update with a
workspace, through the C-ABI: two calls in a row on one GPU, the second on
a smaller input, each compared bit for bit (same kernels and summation
order). The first input has segments long enough to be split into pieces
(Zipf hot rows), so the scratch's work lists, piece sums and counters are
used; the second call must not see the first call's leftovers. Also: the
size limit is enforced before anything is launched."""
import numpy as np
import pytest
import torch

from paper_2010_13100_amd import tc
from paper_2010_13100_amd import workload as wl
from tests.gpu_harness import DeviceRun, assert_close, to_dev

pytestmark = pytest.mark.gpu

W = wl.WORKLOADS
BIG = W["c5"].scaled(name="c5-1x200k", num_tables=1, rows_per_table=200_000, batch=509)
SMALL = W["c2"].scaled(name="c2-2x20k-b200", num_tables=2, rows_per_table=20_000, batch=200,
                       optimizer="adagrad")


def cast_and_grad(run, b):
    t = run.trainer
    t.cast(to_dev(b.table_row_offset), to_dev(b.indices), to_dev(b.bag_offsets), b.num_pairs)
    return to_dev(b.grad_out)


def test_noalloc_matches_workspace_call_twice():
    for w, step in ((BIG, 0), (SMALL, 1)):
        b = wl.make_batch(w, step)
        print(f"\n[noalloc] {w.name}: {b.num_pairs} pairs", flush=True)
        assert tc.tc_backward_workspace_bytes(b.num_pairs, w.dim) <= tc.TC_NOALLOC_SCRATCH_BYTES
        ref = DeviceRun(w, max_pairs=b.num_pairs, split_long=True)
        got = DeviceRun(w, max_pairs=b.num_pairs, split_long=False)
        for r in (ref, got):
            g = cast_and_grad(r, b)
        t_ref, t_got = ref.trainer, got.trainer
        t_ref.backward_update(g, store_coal=True)
        tc.tc_embed_backward_update_noalloc(
            g, t_got.seg_offsets, t_got.casted_src, t_got.unique_rows, t_got.num_unique,
            t_got.max_unique, b.num_pairs, t_got.W, t_got.A, t_got.opt_kind, t_got.lr, t_got.eps,
            t_got.gamma, t_got.coal)
        torch.cuda.synchronize()
        u = int(t_ref.num_unique.item())
        assert u == int(t_got.num_unique.item())
        so = t_ref.seg_offsets[:u + 1].cpu().numpy()
        longest = int(np.diff(so).max())
        print(f"[noalloc] {u} coalesced rows, longest segment {longest}", flush=True)
        if w is BIG:
            assert longest >= 2048          # the scratch's piece lists are used
        assert_close(t_got.coal[:u].cpu().numpy(), t_ref.coal[:u].cpu().numpy(),
                     "coalesced rows", bitwise=True)
        assert torch.equal(t_got.W, t_ref.W)
        if t_ref.A is not None:
            assert torch.equal(t_got.A, t_ref.A)
        ref.release()
        got.release()


@pytest.mark.parametrize("dim,opt", [(4, "sgd"), (260, "rmsprop"), (1024, "adagrad")])
def test_noalloc_row_shapes_and_optimizers(dim, opt):
    """Every lane-group shape class of the backward (1-lane rows, partial
    float4 chunks over several 64-column parts, 4 chunks per lane) and each
    fused optimizer, with hot rows split into pieces, against the workspace
    call bit for bit."""
    w = W["c2"].scaled(name=f"noalloc-d{dim}", num_tables=2, rows_per_table=5_000, dim=dim,
                       batch=300, optimizer=opt)
    b = wl.make_batch(w, 0)
    ref = DeviceRun(w, max_pairs=b.num_pairs, split_long=True)
    got = DeviceRun(w, max_pairs=b.num_pairs, split_long=False)
    for r in (ref, got):
        g = cast_and_grad(r, b)
    t_ref, t_got = ref.trainer, got.trainer
    t_ref.backward_update(g, store_coal=True)
    tc.tc_embed_backward_update_noalloc(
        g, t_got.seg_offsets, t_got.casted_src, t_got.unique_rows, t_got.num_unique,
        t_got.max_unique, b.num_pairs, t_got.W, t_got.A, t_got.opt_kind, t_got.lr, t_got.eps,
        t_got.gamma, t_got.coal)
    torch.cuda.synchronize()
    u = int(t_ref.num_unique.item())
    so = t_ref.seg_offsets[:u + 1].cpu().numpy()
    assert int(np.diff(so).max()) >= 2048    # some rows are summed in pieces
    assert torch.equal(t_got.coal[:u], t_ref.coal[:u])
    assert torch.equal(t_got.W, t_ref.W)
    if t_ref.A is not None:
        assert torch.equal(t_got.A, t_ref.A)
    ref.release()
    got.release()


def test_noalloc_rejects_oversize_before_launch():
    """More pairs than the scratch covers: TC_ERR_WORKSPACE, nothing touched
    (the buffers are host memory, which a launch would fault on)."""
    lib = tc._lib
    f = np.zeros(64, np.float32)
    i = np.zeros(64, np.int32)
    fp = (f.ctypes.data + 15) // 16 * 16
    big = 40_000_000   # beyond the cover at dim 64
    assert tc.tc_backward_workspace_bytes(big, 64) > tc.TC_NOALLOC_SCRATCH_BYTES
    rc = lib.tc_embed_backward_update_noalloc(fp, 4, 64, i.ctypes.data, i.ctypes.data,
                                              i.ctypes.data, i.ctypes.data, 4, big, fp, None,
                                              16, tc.TC_OPT_SGD, 0.01, 1e-8, 0.0, None, None)
    assert rc == tc.TC_ERR_WORKSPACE
    assert "scratch" in lib.tc_last_error().decode()
    assert not f.any() and not i.any()
