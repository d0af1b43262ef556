"""The long-segment chains when the gathered array is larger than a 32-bit
buffer window (about 2 GiB).

A long segment's rows are loaded through a buffer resource. When the whole
gradient array (grad_out for Algorithm 3, the expanded array for Algorithm
1's accumulate) fits in the window, rows are addressed from its start; when
it does not, a chain whose rows span less than the window is addressed from
its first row, and a chain whose rows span more falls back to 64-bit
addressed loads. This test builds a 2.4 GB grad_out (600k bags of 1024
floats) and a batch whose hot rows hit each case, with and without the
backward workspace (split pieces and whole segments), and checks:

  - tc_embed_backward with a workspace against the fp32 oracle's
    Algorithm 3 (split rows in the documented piece order), bit for bit;
  - tc_embed_backward without a workspace against the oracle's sequential
    sums, bit for bit;
  - tc_embed_coalesce over the 2.5 GB expanded array (tc_embed_expand,
    tc_argsort_rows) equal to the casted backward bit for bit.

Every hot row is checked, plus 2000 random coalesced rows.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2010_13100_amd import tc
from tests.gpu_harness import SPLIT_PAIRS, assert_close, piecewise_row, to_dev

pytestmark = pytest.mark.gpu

ROWS, DIM, BAGS = 1_000_000, 1024, 600_000
WINDOW = 0x7FFFF000  # bytes a chain's rows may span in one buffer window


def build_batch(seed=11):
    """(indices, bag_offsets, grad_out, hot rows). One table; every bag has
    one uniform filler pair, and hot rows add pairs to chosen bags."""
    rng = np.random.default_rng(seed)
    hot = {
        # split, every piece within a window: 3000 pairs in 3000 nearby bags
        11: np.arange(200_000, 203_000),
        # split, first piece spanning more than the window (bag 0 and bags
        # from 597000), second piece within one: 2100 pairs, 2 pieces
        12: np.concatenate([[0], np.arange(597_000, 599_099)]),
        # split, first piece within a window, second one spanning more than
        # the window (it ends at the last bag): 2200 pairs, 2 pieces
        13: np.concatenate([np.arange(0, 2199), [BAGS - 1]]),
        # long, not split, rows within a window
        14: np.arange(100_000, 100_500),
        # long, not split, rows spanning more than the window
        15: np.linspace(0, BAGS - 1, 500).astype(np.int64),
        # long, just under the split length, spanning more than the window
        16: np.linspace(3, BAGS - 2, SPLIT_PAIRS - 1).astype(np.int64),
    }
    hot_rows = np.array(sorted(hot), np.int64)
    filler = rng.integers(100, ROWS, size=BAGS)
    bags = np.concatenate([np.arange(BAGS)] + [hot[r] for r in hot_rows])
    rows = np.concatenate([filler] + [np.full(len(hot[r]), r) for r in hot_rows])
    order = np.argsort(bags, kind="stable")
    bags, rows = bags[order], rows[order]
    offsets = np.concatenate([[0], np.cumsum(np.bincount(bags, minlength=BAGS))])
    grad = rng.standard_normal((BAGS, DIM), dtype=np.float32)
    assert grad.nbytes > WINDOW
    return rows.astype(np.int32), offsets.astype(np.int32), grad, hot_rows


def test_chains_beyond_a_32bit_window():
    idx, bo, grad, hot_rows = build_batch()
    n = len(idx)
    print(f"\n[large grad] {n} pairs, grad_out {grad.nbytes / 2**30:.2f} GiB", flush=True)
    dev = dict(device="cuda")
    i32 = dict(dtype=torch.int32, device="cuda")
    off = to_dev(np.array([0, ROWS], np.int64))
    d_idx, d_bo, d_grad = to_dev(idx), to_dev(bo), to_dev(grad)
    max_unique = min(n, ROWS)
    unique_rows = torch.empty(max_unique, **i32)
    seg = torch.empty(max_unique + 1, **i32)
    casted_src = torch.empty(n, **i32)
    nu = torch.zeros(1, **i32)
    ws = torch.empty(max(tc.tc_cast_workspace_bytes(n, ROWS, 1), 256), dtype=torch.uint8, **dev)
    bws = torch.empty(tc.tc_backward_workspace_bytes(n, DIM), dtype=torch.uint8, **dev)
    tc.tc_cast_index(off, 1, BAGS, ROWS, ROWS, d_idx, d_bo, n, unique_rows, seg, casted_src,
                     None, nu, ws)
    coal_ws = torch.empty((max_unique, DIM), dtype=torch.float32, **dev)
    tc.tc_embed_backward(d_grad, seg, casted_src, nu, max_unique, coal_ws, bws)
    coal_chain = torch.empty_like(coal_ws)
    tc.tc_embed_backward(d_grad, seg, casted_src, nu, max_unique, coal_chain, None)
    torch.cuda.synchronize()
    print("[large grad] casted backward done (with and without workspace)", flush=True)

    # the oracle: Algorithm 2 for the index outputs, Algorithm 3 per row
    orc = oracle.Oracle("f32")
    src = idx.astype(np.int64)
    dst = np.repeat(np.arange(BAGS), np.diff(bo)).astype(np.int32)
    ref = orc.tensor_casting(src, dst)
    u = int(nu.item())
    assert u == ref["num_unique"]
    assert np.array_equal(unique_rows[:u].cpu().numpy(), ref["unique_rows"])
    so = ref["seg_offsets"]
    assert np.array_equal(seg[:u + 1].cpu().numpy(), so)
    assert np.array_equal(casted_src[:n].cpu().numpy(), ref["casted_src"])
    cs = ref["casted_src"]

    rng = np.random.default_rng(3)
    hot_u = np.searchsorted(ref["unique_rows"], hot_rows)
    assert np.array_equal(ref["unique_rows"][hot_u], hot_rows)
    pick = np.unique(np.concatenate([hot_u, rng.choice(u, size=2000, replace=False)]))
    spans = []
    for k in hot_u:
        b = cs[so[k]:so[k + 1]]
        spans.append((so[k + 1] - so[k], (int(b[-1]) - int(b[0]) + 1) * DIM * 4 > WINDOW))
    print(f"[large grad] hot segments (length, spans past the window): {spans}", flush=True)
    assert any(s for _, s in spans) and not all(s for _, s in spans)

    seq = np.stack([orc.casted_gather_reduce(cs[so[k]:so[k + 1]],
                                             np.zeros(so[k + 1] - so[k], np.int32), grad, 1)[0]
                    for k in pick])
    split = np.stack([piecewise_row(orc, cs[so[k]:so[k + 1]], grad)
                      if so[k + 1] - so[k] >= SPLIT_PAIRS else seq[i]
                      for i, k in enumerate(pick)])
    sel = torch.from_numpy(pick).cuda()
    got_ws = coal_ws.index_select(0, sel).cpu().numpy()
    got_chain = coal_chain.index_select(0, sel).cpu().numpy()
    assert_close(got_ws, split, "backward with workspace (pieces)", bitwise=True)
    assert_close(got_chain, seq, "backward without workspace (one chain)", bitwise=True)

    # Algorithm 1's accumulate over the expanded array (2.5 GB)
    del d_grad
    expanded = torch.empty((n, DIM), dtype=torch.float32, **dev)
    assert expanded.numel() * 4 > WINDOW
    tc.tc_embed_expand(to_dev(grad), d_bo, n, expanded)
    sorted_pos = torch.empty(n, **i32)
    seg2 = torch.empty_like(seg)
    nu2 = torch.zeros(1, **i32)
    tc.tc_argsort_rows(off, 1, BAGS, ROWS, ROWS, d_idx, d_bo, n, unique_rows, seg2, sorted_pos,
                       nu2, ws)
    coal_base = torch.empty_like(coal_ws)
    tc.tc_embed_coalesce(expanded, n, seg2, sorted_pos, nu2, max_unique, coal_base, bws)
    torch.cuda.synchronize()
    assert int(nu2.item()) == u
    assert torch.equal(coal_base[:u], coal_ws[:u])
    print("[large grad] expand-coalesce equals the casted backward", flush=True)
