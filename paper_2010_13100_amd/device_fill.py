"""Binding of libtc_workload (include/tc_workload.h): fill a synthetic table
on the GPU with the same SplitMix64 values ``workload.table_rows`` computes
on the host."""
from __future__ import annotations

import ctypes
import os

import torch

from . import build as _build

_path = _build.lib_path("libtc_workload.so")
if not os.path.exists(_path):
    raise ImportError(f"libtc_workload not built: {_path} is missing")
_lib = ctypes.CDLL(_path)
_lib.tcw_fill_uniform.restype = ctypes.c_int
_lib.tcw_fill_uniform.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_uint64, ctypes.c_float, ctypes.c_float, ctypes.c_void_p]


def fill_uniform(W: torch.Tensor, *, seed: int = 0, lo: float = -0.01, hi: float = 0.01,
                 row_begin: int = 0, stream=None) -> None:
    """Fill the rows of ``W`` (rows ``row_begin..`` of the concatenated table)."""
    assert W.is_cuda and W.dtype == torch.float32 and W.is_contiguous() and W.dim() == 2
    s = (stream or torch.cuda.current_stream()).cuda_stream
    # W's first row is global row `row_begin`; the kernel indexes from row 0.
    base = W.data_ptr() - row_begin * W.shape[1] * 4
    rc = _lib.tcw_fill_uniform(base, row_begin, W.shape[0], W.shape[1], seed, lo, hi, s)
    if rc != 0:
        raise RuntimeError(f"tcw_fill_uniform failed ({rc})")
