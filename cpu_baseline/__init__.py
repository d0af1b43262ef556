"""Multi-threaded CPU baseline of the training step (OpenMP over all host
cores): the paper's baseline backward (expand, stable argsort, Algorithm 1)
with the forward and the update, as a reported baseline for the benchmark.

Not the product and not the oracle: only ``bench.py`` and ``tests/`` use it,
it shares no code with the HIP library or the oracle, and its outputs equal
the single-threaded oracle's bit for bit (tests/test_cpu_baseline.py). This
module compiles ``tc_cpu_omp.c`` with gcc and marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tc_cpu_omp.c")
_LIB = os.path.join(_HERE, "libtc_cpu_omp.so")
_CFLAGS = ["-O3", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> None:
    cmd = ["gcc", *_CFLAGS, _SRC, "-o", _LIB, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)


def _lib():
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.cpu_train_step.restype = ctypes.c_int64
    lib.cpu_train_step.argtypes = [i32, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp, i32,
                                   ctypes.c_float, ctypes.c_float, vp]
    lib.cpu_threads.restype = ctypes.c_int
    return lib


class CpuBaseline:
    def __init__(self):
        self.lib = _lib()

    @property
    def threads(self) -> int:
        return int(self.lib.cpu_threads())

    def train_step(self, bag_offsets, pair_row, table, grad_out, optimizer="sgd", acc=None,
                   lr=np.float32(0.01), eps=np.float32(1e-8)):
        """One step on a row set. pair_row[j]: row of pair j in `table` (fp32,
        updated in place, as `acc` for Adagrad). Returns (out, coal, coal_rows,
        seconds per phase: forward, expand, sort, coalesce, update)."""
        bo = np.ascontiguousarray(bag_offsets, np.int32)
        pr = np.ascontiguousarray(pair_row, np.int32)
        g = np.ascontiguousarray(grad_out, np.float32)
        assert table.dtype == np.float32 and table.flags.c_contiguous
        nb, dim = len(bo) - 1, table.shape[1]
        n = int(bo[-1])
        opt = {"sgd": 0, "adagrad": 1}[optimizer]
        if opt == 1:
            assert acc is not None and acc.dtype == np.float32 and acc.shape == table.shape
        out = np.empty((nb, dim), np.float32)
        coal = np.empty((max(n, 1), dim), np.float32)
        rows = np.empty(max(n, 1), np.int32)
        sec = np.zeros(5, np.float64)
        u = self.lib.cpu_train_step(nb, bo.ctypes.data, pr.ctypes.data, table.shape[0], dim,
                                    table.ctypes.data, None if acc is None else acc.ctypes.data,
                                    g.ctypes.data, out.ctypes.data, coal.ctypes.data,
                                    rows.ctypes.data, opt, float(lr), float(eps),
                                    sec.ctypes.data)
        if u < 0:
            raise RuntimeError(f"cpu_train_step failed with code {u}")
        phases = dict(zip(("forward", "expand", "sort", "coalesce", "update"), sec.tolist()))
        return out, coal[:u], rows[:u], phases
