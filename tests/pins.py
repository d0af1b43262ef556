"""Pins that tie the CPU oracle to what the paper and plain mathematics fix.

Every pin takes an ``oracle.Oracle`` and raises ``AssertionError`` (or
``oracle.OracleError``) when the oracle disagrees. None of them re-types the
oracle's loops: they check against a dense matrix product, Python's own
``sorted``, a printed worked example, exact closed forms of one optimizer
step, invariants, brute force over tiny inputs, and a-priori rounding-error
bounds. ``test_oracle_pins.py`` runs them on both oracle builds and
``test_oracle_mutations.py`` checks that planted mistakes trip them.
"""
from __future__ import annotations

import itertools
import os

import numpy as np

from paper_2010_13100_amd import workload as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
U32 = 2.0 ** -24
U64 = 2.0 ** -53


# ----------------------------------------------------------------------------
# fixtures and independent references
# ----------------------------------------------------------------------------

def load_worked_example() -> dict:
    out = {}
    with open(os.path.join(GOLDEN, "worked_example.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, val = line.split(":", 1)
            if key == "coal_terms":
                out[key] = [[int(x) for x in part.split()] for part in val.split("|")]
            else:
                out[key] = [int(x) for x in val.split()]
    return out


def incidence(src, dst, num_bags, num_rows) -> np.ndarray:
    """Dense bag x row matrix whose entries count the pairs (multiplicity)."""
    a = np.zeros((num_bags, num_rows), dtype=np.float64)
    np.add.at(a, (np.asarray(dst, np.int64), np.asarray(src, np.int64)), 1.0)
    return a


def small_instance(seed: int, *, num_tables=2, rows=40, dim=8, batch=12, pool=5, dist="zipf",
                   alpha=1.1, pooling="fixed"):
    """A tiny bag-major CSR instance drawn by the workload generator."""
    w = wl.Workload("pin", 100 + seed, num_tables, rows, dim, batch, pooling, pool, dist, alpha)
    b = wl.make_batch(w, step=seed)
    return w, b


def gamma(k, u):
    k = np.asarray(k, dtype=np.float64)
    return k * u / (1.0 - k * u)


# ----------------------------------------------------------------------------
# index-level pins
# ----------------------------------------------------------------------------

def pin_worked_example(orc):
    ex = load_worked_example()
    src, dst = orc.pairs_from_csr(ex["num_tables"][0], ex["bags_per_table"][0],
                                  np.array([0, ex["rows"][0]]), np.array(ex["indices"]),
                                  np.array(ex["bag_offsets"]))
    assert src.tolist() == ex["src"] and dst.tolist() == ex["dst"]
    cast = orc.tensor_casting(src, dst)
    assert cast["casted_src"].tolist() == ex["casted_src"]
    assert cast["casted_dst"].tolist() == ex["casted_dst"]
    assert cast["unique_rows"].tolist() == ex["unique_rows"]
    assert cast["seg_offsets"].tolist() == ex["seg_offsets"]
    assert cast["num_unique"] == ex["num_unique"][0]
    sorted_src = [cast["unique_rows"][c] for c in cast["casted_dst"]]
    assert sorted_src == ex["sorted_src"]
    # Float side of the example with integer gradients of our choosing.
    g = np.array([[3.0, -1.0, 0.5, 8.0], [-2.0, 4.0, 0.25, 16.0]])
    coal, rows = orc.coalesce(src, orc.expand(dst, g))
    want = np.stack([g[terms].sum(axis=0) for terms in ex["coal_terms"]])
    assert rows.tolist() == ex["unique_rows"]
    assert np.array_equal(coal, want)
    coal3 = orc.casted_gather_reduce(cast["casted_src"], cast["casted_dst"], g, cast["num_unique"])
    assert np.array_equal(coal3, want)
    # Row 3 is never gathered, so a scatter leaves it untouched.
    tbl = np.arange(20, dtype=orc.dtype).reshape(5, 4)
    before = tbl.copy()
    orc.scatter_sgd(rows, coal, 0.5, tbl)
    for r in ex["untouched_rows"]:
        assert np.array_equal(tbl[r], before[r])


def pin_cast_matches_sorted(orc, seeds=range(6)):
    """Algorithm 2 with a stable sort == Python's sort of the (row, bag) pairs."""
    for seed in seeds:
        w, b = small_instance(seed, dist="zipf" if seed % 2 else "uniform")
        src, dst = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                      b.bag_offsets)
        cast = orc.tensor_casting(src, dst)
        ordered = sorted(zip(src.tolist(), dst.tolist()))
        assert cast["casted_src"].tolist() == [d for _, d in ordered]
        uniq = sorted(set(src.tolist()))
        assert cast["unique_rows"].tolist() == uniq
        assert cast["casted_dst"].tolist() == [uniq.index(s) for s, _ in ordered]


def pin_cast_invariants(orc, seeds=range(4)):
    for seed in seeds:
        w, b = small_instance(seed, rows=30, batch=20, pool=7, alpha=1.3)
        src, dst = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                      b.bag_offsets)
        c = orc.tensor_casting(src, dst)
        n, u = len(src), c["num_unique"]
        ur, so, cs, cd = c["unique_rows"], c["seg_offsets"], c["casted_src"], c["casted_dst"]
        assert u == len(np.unique(src))
        assert np.all(np.diff(ur) > 0)                       # strictly increasing rows
        assert so[0] == 0 and so[-1] == n and np.all(np.diff(so) > 0)
        key = ur[cd]                                         # row of every casted pair
        # the casted pairs are a permutation of the input pairs (multiset equality)
        got = sorted(zip(key.tolist(), cs.tolist()))
        assert got == sorted(zip(src.tolist(), dst.tolist()))
        assert np.all(np.diff(key) >= 0)
        assert np.all(cd == np.repeat(np.arange(u), np.diff(so)))
        for i in range(u):                                   # bags ascend inside a segment
            assert np.all(np.diff(cs[so[i]:so[i + 1]]) >= 0)


# ----------------------------------------------------------------------------
# float pins against closed forms
# ----------------------------------------------------------------------------

def pin_forward_closed_form(orc, seeds=range(4)):
    """out = A . W with integer-valued W (exact in any order)."""
    for seed in seeds:
        w, b = small_instance(seed, dim=6)
        rng = np.random.default_rng(seed)
        tbl = rng.integers(-9, 10, size=(w.total_rows, w.dim)).astype(np.float64)
        src, dst = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                      b.bag_offsets)
        out = orc.forward(src, dst, w.num_bags, tbl)
        a = incidence(src, dst, w.num_bags, w.total_rows)
        assert np.array_equal(out, a @ tbl)
        # the same through a sparse row set holding only the gathered rows
        ids = np.unique(src)
        out2 = orc.forward(src, dst, w.num_bags, tbl[ids], ids)
        assert np.array_equal(out2, out)
    # bag size one is a plain gather, bit for bit, on random data
    rng = np.random.default_rng(7)
    tbl = rng.standard_normal((50, 8)).astype(np.float32)
    rows = rng.integers(0, 50, size=30)
    out = orc.forward(rows, np.arange(30), 30, tbl)
    assert np.array_equal(out, tbl[rows].astype(orc.dtype))


def pin_backward_closed_form(orc, seeds=range(4)):
    """Coalesced gradients = (A^T . grad_out) on the rows that were gathered."""
    for seed in seeds:
        w, b = small_instance(seed, dim=5, alpha=1.4)
        rng = np.random.default_rng(seed + 11)
        g = rng.integers(-6, 7, size=(w.num_bags, w.dim)).astype(np.float64)
        src, dst = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                      b.bag_offsets)
        a = incidence(src, dst, w.num_bags, w.total_rows)
        gt = a.T @ g
        touched = np.flatnonzero(a.sum(axis=0) > 0)
        coal, rows = orc.coalesce(src, orc.expand(dst, g))
        assert rows.tolist() == touched.tolist()
        assert np.array_equal(coal, gt[touched])
        cast = orc.tensor_casting(src, dst)
        coal3 = orc.casted_gather_reduce(cast["casted_src"], cast["casted_dst"], g,
                                         cast["num_unique"])
        assert np.array_equal(coal3, gt[touched])
        # column-sum invariant: sum_u coal[u] = sum_b L_b * grad_out[b]
        lengths = np.diff(b.bag_offsets).astype(np.float64)
        assert np.array_equal(coal.sum(axis=0), lengths @ g)
    # special cases: every pair on one row, and all rows distinct
    rng = np.random.default_rng(5)
    g = rng.integers(-4, 5, size=(6, 3)).astype(np.float64)
    src = np.full(10, 7, dtype=np.int64)
    dst = np.sort(rng.integers(0, 6, size=10)).astype(np.int32)
    coal, rows = orc.coalesce(src, orc.expand(dst, g))
    assert rows.tolist() == [7] and np.array_equal(coal[0], g[dst].sum(axis=0))
    src = rng.permutation(40)[:10].astype(np.int64)
    coal, rows = orc.coalesce(src, orc.expand(dst, g))
    order = np.argsort(src)
    assert np.array_equal(rows, src[order]) and np.array_equal(coal, g[dst[order]])


def pin_brute_force(orc):
    """Every index layout with 3 rows, 2 bags and bags of 0..2 gathers."""
    rows, dim = 3, 4
    bag_choices = [()] + [(r,) for r in range(rows)] + list(itertools.product(range(rows), repeat=2))
    assert len(bag_choices) == 13
    rng = np.random.default_rng(3)
    tbl = rng.integers(-5, 6, size=(rows, dim)).astype(np.float64)
    g = rng.integers(-5, 6, size=(2, dim)).astype(np.float64)
    for bag0, bag1 in itertools.product(bag_choices, repeat=2):
        idx = np.array(bag0 + bag1, dtype=np.int32)
        off = np.array([0, len(bag0), len(bag0) + len(bag1)], dtype=np.int32)
        src, dst = orc.pairs_from_csr(1, 2, np.array([0, rows]), idx, off)
        a = incidence(src, dst, 2, rows)
        assert np.array_equal(orc.forward(src, dst, 2, tbl), a @ tbl)
        cast = orc.tensor_casting(src, dst)
        ordered = sorted(zip(src.tolist(), dst.tolist()))
        assert cast["casted_src"].tolist() == [d for _, d in ordered]
        touched = np.flatnonzero(a.sum(axis=0) > 0)
        assert cast["unique_rows"].tolist() == touched.tolist()
        coal, crow = orc.coalesce(src, orc.expand(dst, g))
        assert np.array_equal(coal, (a.T @ g)[touched])
        coal3 = orc.casted_gather_reduce(cast["casted_src"], cast["casted_dst"], g,
                                         cast["num_unique"])
        assert np.array_equal(coal3, (a.T @ g)[touched])
        # sparse SGD update == dense update over every row (lr = 0.5, exact)
        t = tbl.astype(orc.dtype).copy()
        orc.scatter_sgd(crow, coal, 0.5, t)
        assert np.array_equal(t, tbl - 0.5 * (a.T @ g))


def pin_alg1_equals_alg3(orc, seeds=range(3)):
    """The casted gather-reduce equals expand + coalesce bit for bit: both add
    the same gradients in the same (stable sorted) order."""
    for seed in seeds:
        w, b = small_instance(seed, rows=200, dim=16, batch=64, pool=9, alpha=1.2)
        src, dst = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                      b.bag_offsets)
        g = b.grad_out
        coal1, _ = orc.coalesce(src, orc.expand(dst, g))
        cast = orc.tensor_casting(src, dst)
        coal3 = orc.casted_gather_reduce(cast["casted_src"], cast["casted_dst"], g,
                                         cast["num_unique"])
        assert np.array_equal(coal1, coal3)


def pin_sgd_closed_form(orc):
    rng = np.random.default_rng(9)
    tbl = rng.integers(-50, 50, size=(10, 4)).astype(np.float64)
    coal = rng.integers(-8, 8, size=(3, 4)).astype(np.float64)
    rows = np.array([1, 4, 9])
    t = tbl.astype(orc.dtype).copy()
    orc.scatter_sgd(rows, coal, 0.25, t)
    want = tbl.copy()
    want[rows] -= 0.25 * coal
    assert np.array_equal(t, want)


def pin_adagrad_closed_form(orc):
    """Eq. (2) from A = 0 with eps + G^2 a perfect square, so every value is
    exact: G = 0.75, eps = 0.4375 -> sqrt(1) = 1 and W1 = W0 - lr * 0.75."""
    lr, eps = 0.5, 0.4375
    tbl = np.array([[1.0, 2.0, -3.0, 0.0], [4.0, 5.0, 6.0, 7.0], [8.0, 8.5, 9.0, 9.5]])
    coal = np.array([[0.75, -0.75, 0.0, 0.75], [-0.75, 0.75, 0.75, -0.75]])
    rows = np.array([0, 2])
    t, a = tbl.astype(orc.dtype).copy(), np.zeros_like(tbl, dtype=orc.dtype)
    orc.scatter_adagrad(rows, coal, lr, eps, t, a)
    want_t = tbl.copy()
    want_t[rows] -= lr * coal               # G / sqrt(eps + G^2) = G / 1
    want_a = np.zeros_like(tbl)
    want_a[rows] = coal ** 2
    assert np.array_equal(t, want_t) and np.array_equal(a, want_a)
    # second step: A = 0.5625 + G2^2 with G2 = 1.5 gives eps + A = 3.25
    coal2 = np.array([[1.5, 1.5, 1.5, 1.5], [-1.5, 0.0, 1.5, 0.0]])
    orc.scatter_adagrad(rows, coal2, lr, eps, t, a)
    a2 = want_a.copy()
    a2[rows] += coal2 ** 2
    t2 = want_t.copy()
    t2[rows] -= lr * coal2 / np.sqrt(eps + a2[rows])
    tol = 4e-7 if orc.dtype == np.float32 else 1e-15
    assert np.allclose(a, a2, rtol=0, atol=0)
    assert np.allclose(t, t2, rtol=tol, atol=tol)



def pin_rmsprop_special_cases(orc):
    """Eq. (1) at its two ends and at a dyadic middle point, all exact:
    gamma = 0 forgets the past (A = G^2), so one step equals Adagrad's first
    step from A = 0; gamma = 1 keeps A, so W moves by lr*G/sqrt(eps + A0);
    gamma = 0.75 with A0 = 4, G = 2 gives A = 3 + 1 = 4 (a fixed point)."""
    lr = 0.5
    tbl = np.array([[1.0, 2.0, -3.0, 0.0], [4.0, 5.0, 6.0, 7.0], [8.0, 8.5, 9.0, 9.5]])
    rows = np.array([0, 2])
    coal = np.array([[0.75, -0.75, 0.0, 0.75], [-0.75, 0.75, 0.75, -0.75]])
    # gamma = 0 against the Adagrad routine, from a non-zero A0 it must ignore
    eps = 0.4375
    t_r, a_r = tbl.astype(orc.dtype).copy(), np.full(tbl.shape, 9.0, orc.dtype)
    orc.scatter_rmsprop(rows, coal, lr, eps, 0.0, t_r, a_r)
    t_a, a_a = tbl.astype(orc.dtype).copy(), np.zeros(tbl.shape, orc.dtype)
    orc.scatter_adagrad(rows, coal, lr, eps, t_a, a_a)
    a_a[1] = 9.0                            # the untouched row keeps its A
    assert np.array_equal(t_r, t_a) and np.array_equal(a_r, a_a)
    want = tbl.copy()
    want[rows] -= lr * coal                 # eps + G^2 = 1
    assert np.array_equal(t_r, want)
    # gamma = 1: A unchanged (eps + A0 = 4), W -= lr * G / 2
    eps = 1.75
    a0 = np.full(tbl.shape, 2.25)
    t, a = tbl.astype(orc.dtype).copy(), a0.astype(orc.dtype).copy()
    orc.scatter_rmsprop(rows, coal, lr, eps, 1.0, t, a)
    want = tbl.copy()
    want[rows] -= lr * coal / 2
    assert np.array_equal(t, want) and np.array_equal(a, a0)
    # gamma = 0.75, A0 = 4, |G| = 2: A stays 4; eps = 5 -> sqrt(9) = 3
    g2 = np.array([[2.0, -2.0, 2.0, -2.0], [-2.0, 2.0, 2.0, 2.0]])
    a0 = np.full(tbl.shape, 4.0)
    a0[1] = 1.0
    t, a = tbl.astype(orc.dtype).copy(), a0.astype(orc.dtype).copy()
    orc.scatter_rmsprop(rows, g2, 0.75, 5.0, 0.75, t, a)
    want = tbl.copy()
    want[rows] -= 0.75 * g2 / 3             # 0.75 * (+-2/3) = +-0.5 up to rounding
    assert np.array_equal(a, a0)
    tol = 6e-7 if orc.dtype == np.float32 else 2e-15
    assert np.allclose(t, want, rtol=0, atol=tol)


def pin_rmsprop_geometric(orc):
    """k steps of Eq. (1) from A = 0 with a constant gradient G give the
    geometric-series closed form A_k = (1 - gamma^k) G^2, and W moves by
    lr * G * sum_i 1 / sqrt(eps + A_i). gamma = 0.9 is not symmetric, so a
    swap of gamma and 1 - gamma gives (1 - 0.1^k) G^2 instead."""
    gamma, lr, eps, k = 0.9, 0.01, 1e-3, 6
    G = np.array([[0.5, -1.25, 3.0], [2.0, 0.0, -0.125]])
    rows = np.array([1, 3])
    tbl = np.arange(15, dtype=np.float64).reshape(5, 3) * 0.25
    t, a = tbl.astype(orc.dtype).copy(), np.zeros(tbl.shape, orc.dtype)
    want_t = tbl.copy()
    for i in range(1, k + 1):
        orc.scatter_rmsprop(rows, G, lr, eps, gamma, t, a)
        a_i = (1 - gamma ** i) * G ** 2
        want_t[rows] -= lr * G / np.sqrt(eps + a_i)
    tol = 5e-6 if orc.dtype == np.float32 else 1e-13
    assert np.allclose(a[rows], (1 - gamma ** k) * G ** 2, rtol=tol, atol=tol)
    assert np.allclose(t, want_t, rtol=tol, atol=tol)
    untouched = np.setdiff1d(np.arange(5), rows)
    assert np.array_equal(t[untouched], tbl[untouched].astype(orc.dtype))
    assert not np.any(a[untouched])


def pin_rowwise_adagrad_special_cases(orc):
    """Row-wise Adagrad: with dim = 1 it is elementwise Adagrad (the Adagrad
    routine, bit for bit, over two steps); when every column of a row has the
    same |G| the row mean is G^2 and it is elementwise Adagrad again; and
    G = (2, 0, 0, 0) has mean 1, so with eps = 3 the step is G / 2 exactly."""
    lr, eps = 0.5, 0.4375
    rows = np.array([0, 2, 3])
    # dim = 1
    tbl = np.array([[1.0], [2.0], [-3.0], [0.5]])
    t_r, a_r = tbl.astype(orc.dtype).copy(), np.zeros(4, orc.dtype)
    t_e, a_e = tbl.astype(orc.dtype).copy(), np.zeros((4, 1), orc.dtype)
    for coal in (np.array([[0.75], [-1.5], [0.0]]), np.array([[-2.5], [0.25], [1.0]])):
        orc.scatter_rowwise_adagrad(rows, coal, lr, eps, t_r, a_r)
        orc.scatter_adagrad(rows, coal, lr, eps, t_e, a_e)
        assert np.array_equal(t_r, t_e) and np.array_equal(a_r, a_e[:, 0])
    # equal |G| across a row (mean of 4 equal squares is exact)
    tbl = np.arange(20, dtype=np.float64).reshape(5, 4)
    coal = np.array([[0.75, -0.75, 0.75, 0.75], [-1.5, 1.5, 1.5, -1.5], [0.5, 0.5, -0.5, 0.5]])
    t_r, a_r = tbl.astype(orc.dtype).copy(), np.zeros(5, orc.dtype)
    t_e, a_e = tbl.astype(orc.dtype).copy(), np.zeros((5, 4), orc.dtype)
    orc.scatter_rowwise_adagrad(rows, coal, lr, eps, t_r, a_r)
    orc.scatter_adagrad(rows, coal, lr, eps, t_e, a_e)
    assert np.array_equal(t_r, t_e) and np.array_equal(a_r, a_e[:, 0])
    # mean 1, eps 3: W -= lr * G / 2; then a second step adds its own mean
    t, a = tbl.astype(orc.dtype).copy(), np.zeros(5, orc.dtype)
    g1 = np.array([[2.0, 0, 0, 0], [0, -2.0, 0, 0], [0, 0, 0, 2.0]])
    orc.scatter_rowwise_adagrad(rows, g1, 0.5, 3.0, t, a)
    want = tbl.copy()
    want[rows] -= 0.5 * g1 / 2
    assert np.array_equal(t, want)
    assert np.array_equal(a, np.array([1.0, 0, 1.0, 1.0, 0]))
    # second step: G = (1, 3, 1, 3) has mean 5, A = 6, eps + A = 9
    g2 = np.array([[1.0, 3.0, 1.0, 3.0]] * 3)
    orc.scatter_rowwise_adagrad(rows, g2, 0.5, 3.0, t, a)
    want[rows] -= 0.5 * g2 / 3
    assert np.array_equal(a, np.array([6.0, 0, 6.0, 6.0, 0]))
    tol = 6e-7 * 20 if orc.dtype == np.float32 else 1e-14 * 20
    assert np.allclose(t, want, rtol=0, atol=tol)


# ----------------------------------------------------------------------------
# fp32 oracle against the fp64 oracle: a-priori rounding-error bounds
# ----------------------------------------------------------------------------

def _sum_bound(n, abs_sum, u):
    """Recursive summation of n terms from +0 (first add exact):
    |error| <= gamma_{n-1} * sum |x_i|  (Higham, Accuracy and Stability of
    Numerical Algorithms, 2nd ed., eq. 4.4)."""
    return gamma(np.maximum(n - 1, 0), u) * abs_sum


def check_f32_against_f64(orc32, orc64, w: wl.Workload, b: wl.Batch):
    """Every f32 oracle output lies within the rounding-error bound of the
    f64 oracle's value (which is itself within a far smaller bound of the
    exact result)."""
    src, dst = orc64.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                    b.bag_offsets)
    ids = np.unique(src)
    tbl = wl.table_rows(w, ids)
    # forward
    o64 = orc64.forward(src, dst, w.num_bags, tbl, ids)
    o32 = orc32.forward(src, dst, w.num_bags, tbl, ids)
    abs_out = orc64.forward(src, dst, w.num_bags, np.abs(tbl.astype(np.float64)), ids)
    lens = np.diff(b.bag_offsets).astype(np.float64)[:, None]
    bound = _sum_bound(lens, abs_out, U32) + 2 * _sum_bound(lens, abs_out, U64)
    assert np.all(np.abs(o32 - o64) <= bound)
    # backward
    g = b.grad_out
    c64, rows = orc64.coalesce(src, orc64.expand(dst, g))
    c32, rows32 = orc32.coalesce(src, orc32.expand(dst, g))
    assert np.array_equal(rows, rows32)
    a_abs, _ = orc64.coalesce(src, orc64.expand(dst, np.abs(g.astype(np.float64))))
    cnt = np.bincount(np.searchsorted(rows, src), minlength=len(rows)).astype(np.float64)[:, None]
    e_g = _sum_bound(cnt, a_abs, U32) + 2 * _sum_bound(cnt, a_abs, U64)
    assert np.all(np.abs(c32 - c64) <= e_g)
    # SGD from the respective coalesced gradients: W' = W - lr*G with
    # |dW'| <= lr*e_G + u*|lr*G| + u*|W'| (two roundings), first order
    lr = float(np.float32(w.lr))
    t64 = tbl.astype(np.float64).copy()
    t32 = tbl.copy()
    orc64.scatter_sgd(rows, c64, lr, t64, ids)
    orc32.scatter_sgd(rows, c32, lr, t32, ids)
    pos = np.searchsorted(ids, rows)
    e_w = (lr * e_g + U32 * np.abs(lr * c64) + U32 * np.abs(t64[pos])) * (1 + 1e-6) + 1e-30
    assert np.all(np.abs(t32[pos] - t64[pos]) <= e_w)
    # Adagrad from A = 0, propagated to first order through
    # A = G^2, s = sqrt(eps + A), q = G / s, W' = W - lr*q
    eps = float(np.float32(w.eps))
    t64 = tbl.astype(np.float64).copy()
    a64 = np.zeros_like(t64)
    t32 = tbl.copy()
    a32 = np.zeros_like(t32)
    orc64.scatter_adagrad(rows, c64, lr, eps, t64, a64, ids)
    orc32.scatter_adagrad(rows, c32, lr, eps, t32, a32, ids)
    G = np.abs(c64)
    A = a64[pos]
    e_a = 2 * G * e_g + e_g ** 2 + 2 * U32 * A
    s = np.sqrt(eps + A)
    e_s = e_a / (2 * s) + 2 * U32 * s
    q = G / s
    e_q = e_g / s + G * e_s / s ** 2 + U32 * q
    e_w2 = (lr * e_q + U32 * lr * q + U32 * np.abs(t64[pos])) * 1.01 + 1e-30
    assert np.all(np.abs(a32[pos] - A) <= e_a * 1.01 + 1e-30)
    assert np.all(np.abs(t32[pos] - t64[pos]) <= e_w2)


def pin_tables_independent(orc, seeds=range(3)):
    """Several tables in one call give what each table gives on its own
    (each table is its own gather-reduce problem, Sec. II-B): forward outputs,
    casted pairs and coalesced gradients of table t match a single-table call
    on table t's rows, with its row ids shifted by the table's first row."""
    for seed in seeds:
        w, b = small_instance(seed, num_tables=3, rows=25, dim=4, batch=7, pool=6, alpha=1.3)
        rng = np.random.default_rng(seed)
        tbl = rng.integers(-9, 10, size=(w.total_rows, w.dim)).astype(np.float64)
        src, dst = orc.pairs_from_csr(w.num_tables, w.batch, b.table_row_offset, b.indices,
                                      b.bag_offsets)
        out = orc.forward(src, dst, w.num_bags, tbl)
        cast = orc.tensor_casting(src, dst)
        coal, rows = orc.coalesce(src, orc.expand(dst, b.grad_out))
        r0 = 0
        for t in range(w.num_tables):
            lo, hi = b.bag_offsets[t * w.batch], b.bag_offsets[(t + 1) * w.batch]
            off_t = (b.bag_offsets[t * w.batch:(t + 1) * w.batch + 1] - lo).astype(np.int32)
            first = int(b.table_row_offset[t])
            s1, d1 = orc.pairs_from_csr(1, w.batch, np.array([0, w.rows_per_table]),
                                        b.indices[lo:hi], off_t)
            assert np.array_equal(orc.forward(s1, d1, w.batch, tbl[first:first + w.rows_per_table]),
                                  out[t * w.batch:(t + 1) * w.batch])
            c1 = orc.tensor_casting(s1, d1)
            u1 = c1["num_unique"]
            assert np.array_equal(c1["unique_rows"] + first, cast["unique_rows"][r0:r0 + u1])
            assert np.array_equal(c1["casted_src"] + t * w.batch, cast["casted_src"][lo:hi])
            k1, _ = orc.coalesce(s1, orc.expand(d1, b.grad_out[t * w.batch:(t + 1) * w.batch]))
            assert np.array_equal(k1, coal[r0:r0 + u1])
            r0 += u1
        assert r0 == cast["num_unique"] == len(rows)


ALL_PINS = [pin_worked_example, pin_tables_independent, pin_cast_matches_sorted, pin_cast_invariants,
            pin_forward_closed_form, pin_backward_closed_form, pin_brute_force,
            pin_alg1_equals_alg3, pin_sgd_closed_form, pin_adagrad_closed_form,
            pin_rmsprop_special_cases, pin_rmsprop_geometric,
            pin_rowwise_adagrad_special_cases]
