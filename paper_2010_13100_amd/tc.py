"""Python binding of libtc (include/tc.h): argument marshalling only.

Every function has the name of the C entry point it calls and takes torch
tensors that live on the GPU; torch supplies device memory and the stream,
all work runs in the library's HIP kernels. If the library cannot be loaded
the import fails loudly -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

from . import build as _build

TC_OK, TC_ERR_INVALID_ARG, TC_ERR_UNSUPPORTED, TC_ERR_WORKSPACE, TC_ERR_HIP = range(5)
TC_NOALLOC_SCRATCH_BYTES = 16 << 20
TC_INDEX_OK, TC_INDEX_BAD_TABLE_OFFSETS, TC_INDEX_BAD_BAG_OFFSETS, TC_INDEX_OUT_OF_RANGE = range(4)
TC_OPT_SGD, TC_OPT_ADAGRAD, TC_OPT_RMSPROP, TC_OPT_ROWWISE_ADAGRAD = range(4)
OPTIMIZERS = {"sgd": TC_OPT_SGD, "adagrad": TC_OPT_ADAGRAD, "rmsprop": TC_OPT_RMSPROP,
              "rowwise_adagrad": TC_OPT_ROWWISE_ADAGRAD}

_vp, _i32, _i64, _f32, _sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                              ctypes.c_size_t)

_SIGNATURES = {
    "tc_embed_forward": (_i32, [_vp, _i64, _i32, _vp, _i32, _i32, _vp, _vp, _vp, _vp]),
    "tc_cast_workspace_bytes": (_sz, [_i64, _i64, _i32]),
    "tc_cast_index": (_i32, [_vp, _i32, _i32, _i64, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                             _vp, _vp, _sz, _vp]),
    "tc_embed_forward_cast": (_i32, [_vp, _i64, _i32, _vp, _i32, _i32, _i64, _vp, _vp, _i64,
                                     _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "tc_embed_backward": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _i64, _vp, _vp, _sz, _vp]),
    "tc_backward_workspace_bytes": (_sz, [_i64, _i32]),
    "tc_sparse_update": (_i32, [_vp, _vp, _i64, _i32, _vp, _vp, _vp, _i64, _i32, _f32, _f32,
                                _f32, _vp]),
    "tc_embed_backward_update": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _i64, _vp, _vp,
                                        _i64, _i32, _f32, _f32, _f32, _vp, _vp, _sz, _vp]),
    "tc_embed_backward_update_noalloc": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _i64,
                                                _i64, _vp, _vp, _i64, _i32, _f32, _f32, _f32,
                                                _vp, _vp]),
    "tc_argsort_rows": (_i32, [_vp, _i32, _i32, _i64, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                               _vp, _sz, _vp]),
    "tc_embed_expand": (_i32, [_vp, _i32, _i32, _vp, _i64, _vp, _vp]),
    "tc_embed_coalesce": (_i32, [_vp, _i64, _i32, _vp, _vp, _vp, _i64, _vp, _vp, _sz, _vp]),
    "tc_check_index": (_i32, [_vp, _i32, _i32, _i64, _i64, _vp, _vp, _i64, _vp, _vp]),
    "tc_status_string": (ctypes.c_char_p, [_i32]),
    "tc_last_error": (ctypes.c_char_p, []),
    "tc_abi_version": (_i32, []),
}


class TcError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


def load_library(path: str | None = None) -> ctypes.CDLL:
    """libtc.so, or with TC_SANITIZED=1 in the environment the build with the
    host code under AddressSanitizer and UBSan (libtc_san.so; the process
    must preload the sanitizer runtime)."""
    san = os.environ.get("TC_SANITIZED") == "1"
    path = path or _build.lib_path("libtc_san.so" if san else "libtc.so")
    if not os.path.exists(path):
        raise ImportError(f"libtc not built: {path} is missing (run __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    return lib


_lib = load_library()
LIB_PATH = _build.lib_path("libtc.so")


def _ptr(t: torch.Tensor | None, dtype=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check(status: int, what: str) -> None:
    if status != TC_OK:
        name = _lib.tc_status_string(status).decode()
        raise TcError(status, f"{what}: {name}: {_lib.tc_last_error().decode()}")


def tc_abi_version() -> int:
    return int(_lib.tc_abi_version())


def tc_embed_forward(W, table_row_offset, num_tables, bags_per_table, indices, bag_offsets, out,
                     stream=None) -> None:
    _check(_lib.tc_embed_forward(
        _ptr(W, torch.float32, "W"), W.shape[0], W.shape[1],
        _ptr(table_row_offset, torch.int64, "table_row_offset"), num_tables, bags_per_table,
        _ptr(indices, torch.int32, "indices"), _ptr(bag_offsets, torch.int32, "bag_offsets"),
        _ptr(out, torch.float32, "out"), _stream(stream)), "tc_embed_forward")


def tc_cast_workspace_bytes(num_pairs: int, total_rows: int, num_tables: int) -> int:
    return int(_lib.tc_cast_workspace_bytes(num_pairs, total_rows, num_tables))


def tc_cast_index(table_row_offset, num_tables, bags_per_table, total_rows, max_table_rows,
                  indices, bag_offsets, num_pairs, unique_rows, seg_offsets, casted_src,
                  casted_dst, num_unique, workspace, stream=None) -> None:
    _check(_lib.tc_cast_index(
        _ptr(table_row_offset, torch.int64, "table_row_offset"), num_tables, bags_per_table,
        total_rows, max_table_rows, _ptr(indices, torch.int32, "indices"),
        _ptr(bag_offsets, torch.int32, "bag_offsets"), num_pairs,
        _ptr(unique_rows, torch.int32, "unique_rows"), _ptr(seg_offsets, torch.int32, "seg_offsets"),
        _ptr(casted_src, torch.int32, "casted_src"), _ptr(casted_dst, torch.int32, "casted_dst"),
        _ptr(num_unique, torch.int32, "num_unique"), _ptr(workspace, None, "workspace"),
        0 if workspace is None else workspace.numel() * workspace.element_size(),
        _stream(stream)), "tc_cast_index")


def tc_embed_forward_cast(W, table_row_offset, num_tables, bags_per_table, max_table_rows,
                          indices, bag_offsets, num_pairs, out, unique_rows, seg_offsets,
                          casted_src, casted_dst, num_unique, workspace, stream=None) -> None:
    _check(_lib.tc_embed_forward_cast(
        _ptr(W, torch.float32, "W"), W.shape[0], W.shape[1],
        _ptr(table_row_offset, torch.int64, "table_row_offset"), num_tables, bags_per_table,
        max_table_rows, _ptr(indices, torch.int32, "indices"),
        _ptr(bag_offsets, torch.int32, "bag_offsets"), num_pairs,
        _ptr(out, torch.float32, "out"), _ptr(unique_rows, torch.int32, "unique_rows"),
        _ptr(seg_offsets, torch.int32, "seg_offsets"), _ptr(casted_src, torch.int32, "casted_src"),
        _ptr(casted_dst, torch.int32, "casted_dst"), _ptr(num_unique, torch.int32, "num_unique"),
        *_ws(workspace), _stream(stream)), "tc_embed_forward_cast")


def tc_check_index(table_row_offset, num_tables, bags_per_table, total_rows, max_table_rows,
                   indices, bag_offsets, num_pairs, report, stream=None) -> None:
    _check(_lib.tc_check_index(
        _ptr(table_row_offset, torch.int64, "table_row_offset"), num_tables, bags_per_table,
        total_rows, max_table_rows, _ptr(indices, torch.int32, "indices"),
        _ptr(bag_offsets, torch.int32, "bag_offsets"), num_pairs,
        _ptr(report, torch.int64, "report"), _stream(stream)), "tc_check_index")


def _ws(workspace):
    return (_ptr(workspace, None, "workspace"),
            0 if workspace is None else workspace.numel() * workspace.element_size())


def tc_backward_workspace_bytes(num_pairs: int, dim: int) -> int:
    return int(_lib.tc_backward_workspace_bytes(num_pairs, dim))


def tc_embed_backward(grad_out, seg_offsets, casted_src, num_unique, max_unique, coal_grad,
                      workspace=None, stream=None) -> None:
    _check(_lib.tc_embed_backward(
        _ptr(grad_out, torch.float32, "grad_out"), grad_out.shape[0], grad_out.shape[1],
        _ptr(seg_offsets, torch.int32, "seg_offsets"), _ptr(casted_src, torch.int32, "casted_src"),
        _ptr(num_unique, torch.int32, "num_unique"), max_unique,
        _ptr(coal_grad, torch.float32, "coal_grad"), *_ws(workspace), _stream(stream)),
        "tc_embed_backward")


def tc_sparse_update(W, opt_state, unique_rows, coal_grad, num_unique, max_unique, opt_kind, lr,
                     eps, gamma=0.0, stream=None) -> None:
    _check(_lib.tc_sparse_update(
        _ptr(W, torch.float32, "W"), _ptr(opt_state, torch.float32, "opt_state"), W.shape[0],
        W.shape[1], _ptr(unique_rows, torch.int32, "unique_rows"),
        _ptr(coal_grad, torch.float32, "coal_grad"), _ptr(num_unique, torch.int32, "num_unique"),
        max_unique, opt_kind, lr, eps, gamma, _stream(stream)), "tc_sparse_update")


def tc_embed_backward_update(grad_out, seg_offsets, casted_src, unique_rows, num_unique,
                             max_unique, W, opt_state, opt_kind, lr, eps, gamma=0.0,
                             coal_grad=None, workspace=None, stream=None) -> None:
    _check(_lib.tc_embed_backward_update(
        _ptr(grad_out, torch.float32, "grad_out"), grad_out.shape[0], grad_out.shape[1],
        _ptr(seg_offsets, torch.int32, "seg_offsets"), _ptr(casted_src, torch.int32, "casted_src"),
        _ptr(unique_rows, torch.int32, "unique_rows"), _ptr(num_unique, torch.int32, "num_unique"),
        max_unique, _ptr(W, torch.float32, "W"), _ptr(opt_state, torch.float32, "opt_state"),
        W.shape[0], opt_kind, lr, eps, gamma, _ptr(coal_grad, torch.float32, "coal_grad"),
        *_ws(workspace), _stream(stream)), "tc_embed_backward_update")


def tc_embed_backward_update_noalloc(grad_out, seg_offsets, casted_src, unique_rows, num_unique,
                                     max_unique, num_pairs, W, opt_state, opt_kind, lr, eps,
                                     gamma=0.0, coal_grad=None, stream=None) -> None:
    _check(_lib.tc_embed_backward_update_noalloc(
        _ptr(grad_out, torch.float32, "grad_out"), grad_out.shape[0], grad_out.shape[1],
        _ptr(seg_offsets, torch.int32, "seg_offsets"), _ptr(casted_src, torch.int32, "casted_src"),
        _ptr(unique_rows, torch.int32, "unique_rows"), _ptr(num_unique, torch.int32, "num_unique"),
        max_unique, num_pairs, _ptr(W, torch.float32, "W"),
        _ptr(opt_state, torch.float32, "opt_state"), W.shape[0], opt_kind, lr, eps, gamma,
        _ptr(coal_grad, torch.float32, "coal_grad"), _stream(stream)),
        "tc_embed_backward_update_noalloc")


def tc_argsort_rows(table_row_offset, num_tables, bags_per_table, total_rows, max_table_rows,
                    indices, bag_offsets, num_pairs, unique_rows, seg_offsets, sorted_pos,
                    num_unique, workspace, stream=None) -> None:
    _check(_lib.tc_argsort_rows(
        _ptr(table_row_offset, torch.int64, "table_row_offset"), num_tables, bags_per_table,
        total_rows, max_table_rows, _ptr(indices, torch.int32, "indices"),
        _ptr(bag_offsets, torch.int32, "bag_offsets"), num_pairs,
        _ptr(unique_rows, torch.int32, "unique_rows"), _ptr(seg_offsets, torch.int32, "seg_offsets"),
        _ptr(sorted_pos, torch.int32, "sorted_pos"), _ptr(num_unique, torch.int32, "num_unique"),
        _ptr(workspace, None, "workspace"),
        0 if workspace is None else workspace.numel() * workspace.element_size(),
        _stream(stream)), "tc_argsort_rows")


def tc_embed_expand(grad_out, bag_offsets, num_pairs, expanded, stream=None) -> None:
    _check(_lib.tc_embed_expand(
        _ptr(grad_out, torch.float32, "grad_out"), grad_out.shape[0], grad_out.shape[1],
        _ptr(bag_offsets, torch.int32, "bag_offsets"), num_pairs,
        _ptr(expanded, torch.float32, "expanded"), _stream(stream)), "tc_embed_expand")


def tc_embed_coalesce(expanded, num_pairs, seg_offsets, sorted_pos, num_unique, max_unique,
                      coal_grad, workspace=None, stream=None) -> None:
    _check(_lib.tc_embed_coalesce(
        _ptr(expanded, torch.float32, "expanded"), num_pairs, expanded.shape[1],
        _ptr(seg_offsets, torch.int32, "seg_offsets"), _ptr(sorted_pos, torch.int32, "sorted_pos"),
        _ptr(num_unique, torch.int32, "num_unique"), max_unique,
        _ptr(coal_grad, torch.float32, "coal_grad"), *_ws(workspace), _stream(stream)),
        "tc_embed_coalesce")


class EmbeddingTrainer:
    """Device buffers for one workload shape and the calls of a step.

    Buffers are torch tensors (device memory only); the step itself is
    library calls on the current stream (forward and cast, then backward and
    update, each pair one call or two), with no host synchronisation.
    """

    def __init__(self, *, total_rows: int, dim: int, num_tables: int, bags_per_table: int,
                 max_pairs: int, optimizer: str = "sgd", lr: float = 0.01, eps: float = 1e-8,
                 gamma: float = 0.99, device="cuda", table: torch.Tensor | None = None,
                 max_table_rows: int = 0, split_long: bool = True):
        """split_long: give the backward a workspace, so that segments of
        TC_BACKWARD_SPLIT_PAIRS pairs or more are summed in pieces (faster
        under skew; without it every segment is one ordered chain)."""
        self.total_rows, self.dim = total_rows, dim
        self.num_tables, self.bags_per_table = num_tables, bags_per_table
        self.num_bags = num_tables * bags_per_table
        self.max_pairs = max_pairs
        self.max_table_rows = max_table_rows
        self.max_unique = min(max_pairs, total_rows)
        self.opt_kind = OPTIMIZERS[optimizer]
        self.lr, self.eps, self.gamma = lr, eps, gamma
        i32 = dict(dtype=torch.int32, device=device)
        self.W = table if table is not None else torch.empty((total_rows, dim), dtype=torch.float32,
                                                             device=device)
        if self.opt_kind in (TC_OPT_ADAGRAD, TC_OPT_RMSPROP):
            self.A = torch.zeros_like(self.W)
        elif self.opt_kind == TC_OPT_ROWWISE_ADAGRAD:
            self.A = torch.zeros(total_rows, dtype=torch.float32, device=self.W.device)
        else:
            self.A = None
        self.out = torch.empty((self.num_bags, dim), dtype=torch.float32, device=device)
        self.unique_rows = torch.empty(max(self.max_unique, 1), **i32)
        self.seg_offsets = torch.empty(self.max_unique + 1, **i32)
        self.casted_src = torch.empty(max(max_pairs, 1), **i32)
        self.casted_dst = torch.empty(max(max_pairs, 1), **i32)
        self.num_unique = torch.zeros(1, **i32)
        self.coal = torch.empty((max(self.max_unique, 1), dim), dtype=torch.float32, device=device)
        ws = tc_cast_workspace_bytes(max_pairs, total_rows, num_tables)
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=device)
        bws = tc_backward_workspace_bytes(max_pairs, dim) if split_long else 0
        self.bwd_workspace = (torch.empty(bws, dtype=torch.uint8, device=device) if bws
                              else None)
        # cast outputs by slot: slot 0 is the attributes above; cast_slots()
        # adds more, so that the next batch can be cast (on another stream)
        # while a step still reads the current one
        self._slots = [dict(unique_rows=self.unique_rows, seg_offsets=self.seg_offsets,
                            casted_src=self.casted_src, num_unique=self.num_unique)]

    def cast_slots(self, n: int) -> None:
        """Hold n sets of cast outputs (slots 0 .. n-1)."""
        while len(self._slots) < n:
            self._slots.append(dict(unique_rows=torch.empty_like(self.unique_rows),
                                    seg_offsets=torch.empty_like(self.seg_offsets),
                                    casted_src=torch.empty_like(self.casted_src),
                                    num_unique=torch.zeros_like(self.num_unique)))

    def forward(self, table_row_offset, indices, bag_offsets, stream=None):
        tc_embed_forward(self.W, table_row_offset, self.num_tables, self.bags_per_table, indices,
                         bag_offsets, self.out, stream)

    def cast(self, table_row_offset, indices, bag_offsets, num_pairs, stream=None,
             with_casted_dst=False, slot=0):
        c = self._slots[slot]
        tc_cast_index(table_row_offset, self.num_tables, self.bags_per_table, self.total_rows,
                      self.max_table_rows, indices, bag_offsets, num_pairs, c["unique_rows"],
                      c["seg_offsets"], c["casted_src"],
                      self.casted_dst if with_casted_dst else None, c["num_unique"],
                      self.workspace, stream)

    def forward_cast(self, table_row_offset, indices, bag_offsets, num_pairs, stream=None,
                     with_casted_dst=False):
        """forward + cast in one call, overlapped (same results as the two)."""
        tc_embed_forward_cast(self.W, table_row_offset, self.num_tables, self.bags_per_table,
                              self.max_table_rows, indices, bag_offsets, num_pairs, self.out,
                              self.unique_rows, self.seg_offsets, self.casted_src,
                              self.casted_dst if with_casted_dst else None, self.num_unique,
                              self.workspace, stream)

    def backward(self, grad_out, stream=None):
        tc_embed_backward(grad_out, self.seg_offsets, self.casted_src, self.num_unique,
                          self.max_unique, self.coal, self.bwd_workspace, stream)

    def update(self, stream=None):
        tc_sparse_update(self.W, self.A, self.unique_rows, self.coal, self.num_unique,
                         self.max_unique, self.opt_kind, self.lr, self.eps, self.gamma, stream)

    def baseline_backward(self, table_row_offset, indices, bag_offsets, num_pairs, grad_out,
                          stream=None):
        """The paper's baseline backward (expand, stable argsort, Algorithm 1
        accumulate) into self.coal, with the same unique_rows / seg_offsets as
        the cast; needs self.expanded ([max_pairs x dim], allocated here on
        first use) and overwrites casted_src with the sorted positions."""
        if getattr(self, "expanded", None) is None:
            self.expanded = torch.empty((max(self.max_pairs, 1), self.dim), dtype=torch.float32,
                                        device=self.W.device)
        tc_embed_expand(grad_out, bag_offsets, num_pairs, self.expanded, stream)
        tc_argsort_rows(table_row_offset, self.num_tables, self.bags_per_table, self.total_rows,
                        self.max_table_rows, indices, bag_offsets, num_pairs, self.unique_rows,
                        self.seg_offsets, self.casted_src, self.num_unique, self.workspace,
                        stream)
        tc_embed_coalesce(self.expanded, num_pairs, self.seg_offsets, self.casted_src,
                          self.num_unique, self.max_unique, self.coal, self.bwd_workspace,
                          stream)

    def backward_update(self, grad_out, stream=None, store_coal=False, slot=0):
        """backward + update in one pass (coal stored only if store_coal), on
        the cast outputs in `slot`."""
        c = self._slots[slot]
        tc_embed_backward_update(grad_out, c["seg_offsets"], c["casted_src"], c["unique_rows"],
                                 c["num_unique"], self.max_unique, self.W, self.A, self.opt_kind,
                                 self.lr, self.eps, self.gamma,
                                 self.coal if store_coal else None, self.bwd_workspace, stream)

    def step(self, table_row_offset, indices, bag_offsets, num_pairs, grad_out, stream=None,
             fused=True):
        """forward + cast + backward + update, stream-ordered; with fused the
        first two are one overlapped call and the last two one pass
        (row-wise Adagrad always takes the backward and update calls)."""
        if fused:
            self.forward_cast(table_row_offset, indices, bag_offsets, num_pairs, stream)
        else:
            self.forward(table_row_offset, indices, bag_offsets, stream)
            self.cast(table_row_offset, indices, bag_offsets, num_pairs, stream)
        if fused and self.opt_kind != TC_OPT_ROWWISE_ADAGRAD:
            self.backward_update(grad_out, stream)
        else:
            self.backward(grad_out, stream)
            self.update(stream)
