"""CPU oracle for the Tensor Casting training step -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product (``paper_2010_13100_amd``)
never imports it, and it imports nothing from the product.

``tc_oracle.c`` is compiled twice: ``f64`` (double arithmetic, the reference
the pins check against closed forms) and ``f32`` (the same steps in the fp32
arithmetic the workloads fix). Both are plain single-threaded C; this module
only marshals numpy arrays. Functions follow the paper section or algorithm
named in the C source.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tc_oracle.c")
_CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
           "-Wall", "-Wextra"]


# The sanitized builds (TC_SANITIZED=1 in the environment selects them) use
# clang's AddressSanitizer and UndefinedBehaviorSanitizer; the process
# preloads clang's sanitizer runtime (tests/test_sanitizers.py).
_SAN_CC = "/opt/rocm/llvm/bin/clang"
_SAN_FLAGS = ["-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
              "-fno-omit-frame-pointer"]


def sanitized() -> bool:
    return os.environ.get("TC_SANITIZED") == "1"


def lib_path(precision: str, san: bool | None = None) -> str:
    san = sanitized() if san is None else san
    return os.path.join(_HERE, f"liboracle_{precision}{'_san' if san else ''}.so")


def build_one(src: str, precision: str, out: str, verbose: bool = False,
              san: bool = False) -> None:
    """Compile one oracle source for ``precision`` ("f64" or "f32") with gcc
    (or, san=True, with clang and the sanitizers)."""
    ctype = {"f64": "double", "f32": "float"}[precision]
    cc, extra = (_SAN_CC, _SAN_FLAGS) if san else ("gcc", [])
    cmd = [cc, *_CFLAGS, *extra, f"-DOREAL={ctype}", src, "-o", out, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)


def build(verbose: bool = False, san: bool = False) -> None:
    """Compile the f64 and f32 oracle libraries."""
    for prec in ("f64", "f32"):
        build_one(_SRC, prec, lib_path(prec, san), verbose, san)


_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_vp = ctypes.c_void_p


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(_vp)


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str) -> int:
    if rc < 0:
        raise OracleError(f"{what} failed with code {rc}")
    return rc


class Oracle:
    """One build of the oracle library (``precision`` is ``"f64"`` or ``"f32"``)."""

    def __init__(self, precision: str = "f64", path: str | None = None):
        if precision not in ("f64", "f32"):
            raise ValueError(precision)
        if path is None:
            path = lib_path(precision)
            if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
                build(san=sanitized())
        lib = ctypes.CDLL(path)
        self.precision = precision
        self.dtype = np.float64 if precision == "f64" else np.float32
        assert lib.oracle_real_bytes() == np.dtype(self.dtype).itemsize
        vp, i32, i64, dbl = _vp, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        sig = {
            "oracle_pairs_from_csr": (ctypes.c_int, [i32, i32, vp, vp, vp, vp, vp]),
            "oracle_forward": (ctypes.c_int, [i32, i64, vp, vp, i64, vp, i64, vp, vp]),
            "oracle_expand": (ctypes.c_int, [i32, i64, vp, vp, vp]),
            "oracle_coalesce": (i64, [i32, i64, vp, vp, vp, vp]),
            "oracle_tensor_casting": (i64, [i64, vp, vp, vp, vp, vp, vp]),
            "oracle_casted_gather_reduce": (ctypes.c_int, [i32, i64, vp, vp, vp, i64, i64, vp]),
            "oracle_scatter_sgd": (ctypes.c_int, [i32, i64, vp, vp, dbl, vp, i64, vp]),
            "oracle_scatter_adagrad": (ctypes.c_int, [i32, i64, vp, vp, dbl, dbl, vp, i64, vp, vp]),
            "oracle_scatter_rmsprop": (ctypes.c_int,
                                       [i32, i64, vp, vp, dbl, dbl, dbl, vp, i64, vp, vp]),
            "oracle_scatter_rowwise_adagrad": (ctypes.c_int,
                                               [i32, i64, vp, vp, dbl, dbl, vp, i64, vp, vp]),
        }
        for name, (res, args) in sig.items():
            f = getattr(lib, name)
            f.restype, f.argtypes = res, args
        self.lib = lib

    # -- helpers -----------------------------------------------------------
    def _real(self, a) -> np.ndarray:
        return np.ascontiguousarray(a, dtype=self.dtype)

    # -- the index array (Sec. II-B) ---------------------------------------
    def pairs_from_csr(self, num_tables, bags_per_table, table_row_offset, indices, bag_offsets):
        """(src, dst) pairs of the bag-major CSR index array."""
        off = np.ascontiguousarray(table_row_offset, dtype=np.int64)
        idx = np.ascontiguousarray(indices, dtype=np.int32)
        bo = np.ascontiguousarray(bag_offsets, dtype=np.int32)
        n = int(bo[-1]) if len(bo) else 0
        src = np.empty(n, dtype=np.int64)
        dst = np.empty(n, dtype=np.int32)
        _check(self.lib.oracle_pairs_from_csr(num_tables, bags_per_table, _ptr(off), _ptr(idx),
                                              _ptr(bo), _ptr(src), _ptr(dst)), "pairs_from_csr")
        return src, dst

    # -- forward gather-reduce (Sec. II-B) ---------------------------------
    def forward(self, src, dst, num_bags, table, table_ids=None):
        """``out[num_bags, dim]``; ``table`` is dense, or holds the rows ``table_ids``."""
        tbl = self._real(table)
        dim = tbl.shape[1]
        ids = None if table_ids is None else np.ascontiguousarray(table_ids, dtype=np.int64)
        out = np.empty((num_bags, dim), dtype=self.dtype)
        _check(self.lib.oracle_forward(dim, len(src), _ptr(np.ascontiguousarray(src, np.int64)),
                                       _ptr(np.ascontiguousarray(dst, np.int32)), num_bags,
                                       _ptr(ids), tbl.shape[0], _ptr(tbl), _ptr(out)), "forward")
        return out

    # -- baseline backward: expand + coalesce (Sec. II-B, Algorithm 1) -------
    def expand(self, dst, grad_out):
        g = self._real(grad_out)
        dim = g.shape[1]
        exp = np.empty((len(dst), dim), dtype=self.dtype)
        _check(self.lib.oracle_expand(dim, len(dst), _ptr(np.ascontiguousarray(dst, np.int32)),
                                      _ptr(g), _ptr(exp)), "expand")
        return exp

    def coalesce(self, src, expanded):
        """Algorithm 1 -> (coal[U, dim], rows[U])."""
        e = self._real(expanded)
        n, dim = len(src), e.shape[1]
        coal = np.empty((n, dim), dtype=self.dtype)
        rows = np.empty(n, dtype=np.int64)
        u = _check(self.lib.oracle_coalesce(dim, n, _ptr(np.ascontiguousarray(src, np.int64)),
                                            _ptr(e), _ptr(coal), _ptr(rows)), "coalesce")
        return coal[:u].copy(), rows[:u].copy()

    # -- Tensor Casting (Algorithm 2) --------------------------------------
    def tensor_casting(self, src, dst):
        """-> dict(casted_src, casted_dst, unique_rows, seg_offsets, num_unique)."""
        n = len(src)
        cs = np.empty(n, dtype=np.int32)
        cd = np.empty(n, dtype=np.int32)
        ur = np.empty(n, dtype=np.int64)
        so = np.empty(n + 1, dtype=np.int64)
        u = _check(self.lib.oracle_tensor_casting(
            n, _ptr(np.ascontiguousarray(src, np.int64)), _ptr(np.ascontiguousarray(dst, np.int32)),
            _ptr(cs), _ptr(cd), _ptr(ur), _ptr(so)), "tensor_casting")
        return dict(casted_src=cs, casted_dst=cd, unique_rows=ur[:u].copy(),
                    seg_offsets=so[:u + 1].copy(), num_unique=int(u))

    # -- casted gradient gather-reduce (Algorithm 3) -----------------------
    def casted_gather_reduce(self, casted_src, casted_dst, grad_out, num_unique):
        g = self._real(grad_out)
        dim = g.shape[1]
        coal = np.empty((num_unique, dim), dtype=self.dtype)
        _check(self.lib.oracle_casted_gather_reduce(
            dim, len(casted_src), _ptr(np.ascontiguousarray(casted_src, np.int32)),
            _ptr(np.ascontiguousarray(casted_dst, np.int32)), _ptr(g), g.shape[0], num_unique,
            _ptr(coal)), "casted_gather_reduce")
        return coal

    # -- gradient scatter + optimizer (Sec. II-B, Eq. 2) --------------------
    def scatter_sgd(self, rows, coal, lr, table, table_ids=None):
        """Updates ``table`` (an array of this oracle's dtype) in place."""
        assert table.dtype == self.dtype and table.flags.c_contiguous
        c = self._real(coal)
        ids = None if table_ids is None else np.ascontiguousarray(table_ids, dtype=np.int64)
        _check(self.lib.oracle_scatter_sgd(table.shape[1], len(rows),
                                           _ptr(np.ascontiguousarray(rows, np.int64)), _ptr(c),
                                           float(lr), _ptr(ids), table.shape[0], _ptr(table)),
               "scatter_sgd")

    def scatter_adagrad(self, rows, coal, lr, eps, table, acc, table_ids=None):
        """Updates ``table`` and ``acc`` (same row set) in place."""
        assert table.dtype == self.dtype and acc.dtype == self.dtype
        assert table.shape == acc.shape and table.flags.c_contiguous and acc.flags.c_contiguous
        c = self._real(coal)
        ids = None if table_ids is None else np.ascontiguousarray(table_ids, dtype=np.int64)
        _check(self.lib.oracle_scatter_adagrad(table.shape[1], len(rows),
                                               _ptr(np.ascontiguousarray(rows, np.int64)), _ptr(c),
                                               float(lr), float(eps), _ptr(ids), table.shape[0],
                                               _ptr(table), _ptr(acc)), "scatter_adagrad")

    def scatter_rmsprop(self, rows, coal, lr, eps, gamma, table, acc, table_ids=None):
        """Eq. (1); updates ``table`` and ``acc`` (same row set) in place."""
        assert table.dtype == self.dtype and acc.dtype == self.dtype
        assert table.shape == acc.shape and table.flags.c_contiguous and acc.flags.c_contiguous
        c = self._real(coal)
        ids = None if table_ids is None else np.ascontiguousarray(table_ids, dtype=np.int64)
        _check(self.lib.oracle_scatter_rmsprop(table.shape[1], len(rows),
                                               _ptr(np.ascontiguousarray(rows, np.int64)), _ptr(c),
                                               float(lr), float(eps), float(gamma), _ptr(ids),
                                               table.shape[0], _ptr(table), _ptr(acc)),
               "scatter_rmsprop")

    def scatter_rowwise_adagrad(self, rows, coal, lr, eps, table, acc, table_ids=None):
        """Row-wise Adagrad; ``acc`` has one value per stored table row."""
        assert table.dtype == self.dtype and acc.dtype == self.dtype
        assert acc.shape == (table.shape[0],) and table.flags.c_contiguous
        assert acc.flags.c_contiguous
        c = self._real(coal)
        ids = None if table_ids is None else np.ascontiguousarray(table_ids, dtype=np.int64)
        _check(self.lib.oracle_scatter_rowwise_adagrad(
            table.shape[1], len(rows), _ptr(np.ascontiguousarray(rows, np.int64)), _ptr(c),
            float(lr), float(eps), _ptr(ids), table.shape[0], _ptr(table), _ptr(acc)),
            "scatter_rowwise_adagrad")


@dataclass
class StepResult:
    out: np.ndarray            # forward output [T*B, D]
    cast: dict                 # Algorithm 2 outputs
    coal: np.ndarray           # coalesced gradients [U, D] (Algorithm 1)
    coal_rows: np.ndarray      # their table rows [U]
    table: np.ndarray          # updated table rows (same row set as given)
    acc: np.ndarray | None     # updated Adagrad accumulator, or None


def train_step(orc: Oracle, *, num_tables, bags_per_table, table_row_offset, indices, bag_offsets,
               grad_out, table, table_ids=None, optimizer="sgd", lr=0.01, eps=1e-8, acc=None,
               gamma=0.99, timings: dict | None = None) -> StepResult:
    """One oracle training step: forward, the paper's baseline backward
    (expand, then Algorithm 1), Tensor Casting (Algorithm 2) for the index
    outputs, and the scatter update. ``table``/``acc`` are copied, not
    modified. ``timings`` (if given) receives seconds per phase."""
    import time

    def tick(name, t0):
        if timings is not None:
            timings[name] = timings.get(name, 0.0) + time.perf_counter() - t0
        return time.perf_counter()

    t0 = time.perf_counter()
    src, dst = orc.pairs_from_csr(num_tables, bags_per_table, table_row_offset, indices, bag_offsets)
    num_bags = num_tables * bags_per_table
    t0 = tick("pairs", t0)
    out = orc.forward(src, dst, num_bags, table, table_ids)
    t0 = tick("forward", t0)
    cast = orc.tensor_casting(src, dst)
    t0 = tick("cast", t0)
    exp = orc.expand(dst, grad_out)
    t0 = tick("expand", t0)
    coal, rows = orc.coalesce(src, exp)
    del exp
    t0 = tick("coalesce", t0)
    tbl = np.array(table, dtype=orc.dtype, copy=True)
    new_acc = None
    if optimizer == "sgd":
        orc.scatter_sgd(rows, coal, lr, tbl, table_ids)
    elif optimizer == "adagrad":
        new_acc = (np.zeros_like(tbl) if acc is None else np.array(acc, dtype=orc.dtype, copy=True))
        orc.scatter_adagrad(rows, coal, lr, eps, tbl, new_acc, table_ids)
    elif optimizer == "rmsprop":
        new_acc = (np.zeros_like(tbl) if acc is None else np.array(acc, dtype=orc.dtype, copy=True))
        orc.scatter_rmsprop(rows, coal, lr, eps, gamma, tbl, new_acc, table_ids)
    elif optimizer == "rowwise_adagrad":
        new_acc = (np.zeros(tbl.shape[0], orc.dtype) if acc is None
                   else np.array(acc, dtype=orc.dtype, copy=True))
        orc.scatter_rowwise_adagrad(rows, coal, lr, eps, tbl, new_acc, table_ids)
    else:
        raise ValueError(optimizer)
    tick("update", t0)
    return StepResult(out, cast, coal, rows, tbl, new_acc)
