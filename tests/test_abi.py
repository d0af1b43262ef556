"""The C-ABI library on the host: it loads, exports every declared entry
point, and rejects bad arguments before launching anything (no GPU needed)."""
import ctypes
import glob
import os
import re

import numpy as np
import pytest

from paper_2010_13100_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER_LIBS = {"tc.h": "libtc.so", "tc_workload.h": "libtc_workload.so"}


def declared_functions(header: str) -> list:
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tcw?_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def tc():
    from paper_2010_13100_amd import tc as T
    return T


@pytest.mark.parametrize("header", sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))),
                         ids=os.path.basename)
def test_every_declared_symbol_is_exported(header):
    lib = ctypes.CDLL(B.lib_path(HEADER_LIBS[os.path.basename(header)]))
    names = declared_functions(header)
    assert names
    for name in names:
        assert hasattr(lib, name), f"{name} declared in {os.path.basename(header)} but not exported"


def test_version_and_status_strings(tc):
    assert tc.tc_abi_version() == 7
    lib = tc._lib
    for code, name in enumerate(["TC_OK", "TC_ERR_INVALID_ARG", "TC_ERR_UNSUPPORTED",
                                 "TC_ERR_WORKSPACE", "TC_ERR_HIP"]):
        assert lib.tc_status_string(code).decode() == name
    assert lib.tc_status_string(99).decode() == "TC_ERR_UNKNOWN"


def test_backward_workspace_bytes(tc):
    f = tc.tc_backward_workspace_bytes
    assert f(79, 64) == 0 and f(0, 64) == 0 and f(-5, 64) == 0 and f(80, 64) > 0
    assert f(10 ** 6, 0) == 0 and f(10 ** 6, 1028) == 0 and f(2 ** 31, 64) == 0
    sizes = [f(n, 64) for n in (80, 2048, 4096, 10 ** 5, 10 ** 6, 10 ** 7)]
    assert sizes == sorted(sizes) and all(s % 256 == 0 for s in sizes)
    # piece sums (a row of dim floats per 1024 pairs) plus the work lists
    n = 10 ** 7
    assert n // 1024 * 64 * 4 <= f(n, 64) <= n * (64 / 256 + 0.25)
    assert f(10 ** 6, 256) > f(10 ** 6, 64)


def test_workspace_bytes(tc):
    lib = tc._lib
    assert lib.tc_cast_workspace_bytes(-1, 10, 1) == 0
    sizes = [lib.tc_cast_workspace_bytes(n, 1000, 4) for n in (0, 1, 4096, 4097, 10 ** 6)]
    assert sizes == sorted(sizes)
    assert sizes[-1] >= 16 * 10 ** 6   # four int32 arrays of num_pairs
    assert all(s % 256 == 0 for s in sizes)


class HostBuffers:
    """Host arrays standing in for device buffers: validation must fail
    before any of them is read or written."""

    def __init__(self):
        self.f = np.full(4096 + 4, 7.0, dtype=np.float32)
        self.i = np.full(4096, 7, dtype=np.int32)
        self.l = np.full(16, 7, dtype=np.int64)
        self.ws = np.zeros(1 << 16, dtype=np.uint8)

    def fp(self, misalign=False):
        p = self.f.ctypes.data
        p = (p + 15) // 16 * 16
        return p + (4 if misalign else 0)

    def ip(self):
        return self.i.ctypes.data

    def lp(self):
        return self.l.ctypes.data

    def wsp(self, misalign=False):
        p = (self.ws.ctypes.data + 255) // 256 * 256
        return p + (8 if misalign else 0)

    def untouched(self):
        return (np.all(self.f == 7.0) and np.all(self.i == 7) and np.all(self.l == 7)
                and np.all(self.ws == 0))


def _err(tc):
    return tc._lib.tc_last_error().decode()


def test_forward_rejects_bad_arguments(tc):
    lib, h = tc._lib, HostBuffers()
    f = lambda **k: lib.tc_embed_forward(  # noqa: E731
        k.get("W", h.fp()), k.get("rows", 100), k.get("dim", 64), k.get("off", h.lp()),
        k.get("T", 1), k.get("B", 4), k.get("idx", h.ip()), k.get("bo", h.ip()),
        k.get("out", h.fp()), None)
    assert f(dim=6) == tc.TC_ERR_UNSUPPORTED and "multiple of 4" in _err(tc)
    assert f(dim=0) == tc.TC_ERR_UNSUPPORTED
    assert f(dim=2048) == tc.TC_ERR_UNSUPPORTED
    assert f(T=-1) == tc.TC_ERR_INVALID_ARG
    assert f(rows=2 ** 31) == tc.TC_ERR_INVALID_ARG
    assert f(W=None) == tc.TC_ERR_INVALID_ARG and "null" in _err(tc)
    assert f(bo=None) == tc.TC_ERR_INVALID_ARG
    assert f(W=h.fp(misalign=True)) == tc.TC_ERR_UNSUPPORTED
    assert f(T=0) == tc.TC_OK and _err(tc) == ""          # nothing to do, nothing launched
    assert h.untouched()


def test_cast_rejects_bad_arguments(tc):
    lib, h = tc._lib, HostBuffers()
    need = lib.tc_cast_workspace_bytes(1000, 100, 1)

    def f(**k):
        return lib.tc_cast_index(
            k.get("off", h.lp()), k.get("T", 1), k.get("B", 50), k.get("rows", 100),
            k.get("mtr", 100), k.get("idx", h.ip()), k.get("bo", h.ip()), k.get("n", 1000),
            k.get("ur", h.ip()),
            k.get("so", h.ip()), k.get("cs", h.ip()), k.get("cd", None), k.get("nu", h.ip()),
            k.get("ws", h.wsp()), k.get("wsb", need), None)
    assert f(wsb=need - 1) == tc.TC_ERR_WORKSPACE and "workspace" in _err(tc)
    assert f(ws=None) == tc.TC_ERR_WORKSPACE
    assert f(ws=h.wsp(misalign=True)) == tc.TC_ERR_WORKSPACE
    assert f(n=-5) == tc.TC_ERR_INVALID_ARG
    assert f(n=2 ** 31) == tc.TC_ERR_INVALID_ARG
    assert f(rows=2 ** 31) == tc.TC_ERR_INVALID_ARG
    assert f(mtr=-1) == tc.TC_ERR_INVALID_ARG
    assert f(cs=None) == tc.TC_ERR_INVALID_ARG
    assert f(ur=None) == tc.TC_ERR_INVALID_ARG
    assert f(nu=None) == tc.TC_ERR_INVALID_ARG
    assert f(T=0) == tc.TC_ERR_INVALID_ARG     # pairs but no bags
    # the argsort shares the cast's checks, under its own name
    rc = lib.tc_argsort_rows(h.lp(), 1, 50, 100, 100, h.ip(), h.ip(), 1000, h.ip(), h.ip(),
                             h.ip(), h.ip(), h.wsp(), need - 1, None)
    assert rc == tc.TC_ERR_WORKSPACE and "tc_argsort_rows" in _err(tc)
    assert h.untouched()


def test_backward_and_update_reject_bad_arguments(tc):
    lib, h = tc._lib, HostBuffers()

    def bwd(**k):
        return lib.tc_embed_backward(k.get("g", h.fp()), k.get("nb", 10), k.get("dim", 8),
                                     k.get("so", h.ip()), k.get("cs", h.ip()), k.get("nu", h.ip()),
                                     k.get("mu", 10), k.get("coal", h.fp()), k.get("ws", None),
                                     k.get("wsb", 0), None)
    assert bwd(dim=10) == tc.TC_ERR_UNSUPPORTED
    assert bwd(wsb=4096) == tc.TC_ERR_INVALID_ARG and "workspace" in _err(tc)
    assert bwd(ws=h.fp(misalign=True), wsb=4096) == tc.TC_ERR_INVALID_ARG
    assert bwd(mu=-1) == tc.TC_ERR_INVALID_ARG
    assert bwd(nu=None) == tc.TC_ERR_INVALID_ARG
    assert bwd(coal=h.fp(misalign=True)) == tc.TC_ERR_UNSUPPORTED
    assert bwd(mu=0) == tc.TC_OK

    def upd(**k):
        return lib.tc_sparse_update(k.get("W", h.fp()), k.get("A", None), k.get("rows", 100),
                                    k.get("dim", 8), k.get("ur", h.ip()), k.get("coal", h.fp()),
                                    k.get("nu", h.ip()), k.get("mu", 10), k.get("opt", 0),
                                    0.01, 1e-8, k.get("gamma", 0.9), None)
    assert upd(A=h.fp()) == tc.TC_ERR_INVALID_ARG               # SGD takes no state
    assert upd(opt=1) == tc.TC_ERR_INVALID_ARG                  # Adagrad needs state
    assert upd(opt=2) == tc.TC_ERR_INVALID_ARG                  # RMSprop needs state
    assert upd(opt=3) == tc.TC_ERR_INVALID_ARG                  # row-wise Adagrad too
    assert upd(opt=2, A=h.fp(), gamma=1.5) == tc.TC_ERR_INVALID_ARG
    assert upd(opt=2, A=h.fp(), gamma=-0.25) == tc.TC_ERR_INVALID_ARG
    assert upd(opt=2, A=h.fp(), gamma=float("nan")) == tc.TC_ERR_INVALID_ARG
    assert "gamma" in _err(tc)
    assert upd(opt=4, A=h.fp()) == tc.TC_ERR_INVALID_ARG
    assert upd(opt=-1, A=h.fp()) == tc.TC_ERR_INVALID_ARG
    assert upd(opt=2, A=h.fp(misalign=True)) == tc.TC_ERR_UNSUPPORTED
    assert upd(opt=7) == tc.TC_ERR_INVALID_ARG
    assert upd(opt=2, A=h.fp(), mu=0) == tc.TC_OK
    assert upd(dim=3) == tc.TC_ERR_UNSUPPORTED
    assert upd(ur=None) == tc.TC_ERR_INVALID_ARG
    assert upd(opt=1, A=h.fp(misalign=True)) == tc.TC_ERR_UNSUPPORTED

    def fused(**k):
        return lib.tc_embed_backward_update(
            k.get("g", h.fp()), k.get("nb", 10), k.get("dim", 8), k.get("so", h.ip()),
            k.get("cs", h.ip()), k.get("ur", h.ip()), k.get("nu", h.ip()), k.get("mu", 10),
            k.get("W", h.fp()), k.get("A", None), k.get("rows", 100), k.get("opt", 0), 0.01, 1e-8,
            k.get("gamma", 0.9), k.get("coal", None), k.get("ws", None), k.get("wsb", 0), None)
    assert fused(dim=6) == tc.TC_ERR_UNSUPPORTED
    assert fused(mu=-1) == tc.TC_ERR_INVALID_ARG
    assert fused(rows=2 ** 31) == tc.TC_ERR_INVALID_ARG
    assert fused(A=h.fp()) == tc.TC_ERR_INVALID_ARG             # SGD takes no state
    assert fused(opt=1) == tc.TC_ERR_INVALID_ARG                # Adagrad needs state
    assert fused(opt=2) == tc.TC_ERR_INVALID_ARG                # RMSprop needs state
    assert fused(opt=2, A=h.fp(), gamma=2.0) == tc.TC_ERR_INVALID_ARG
    assert fused(opt=3, A=h.fp()) == tc.TC_ERR_UNSUPPORTED      # row-wise: two calls
    assert "row-wise" in _err(tc)
    assert fused(opt=5, A=h.fp()) == tc.TC_ERR_INVALID_ARG
    assert fused(wsb=1024) == tc.TC_ERR_INVALID_ARG
    assert fused(W=None) == tc.TC_ERR_INVALID_ARG and "null" in _err(tc)
    assert fused(ur=None) == tc.TC_ERR_INVALID_ARG
    assert fused(coal=h.fp(misalign=True)) == tc.TC_ERR_UNSUPPORTED
    assert fused(W=h.fp(misalign=True)) == tc.TC_ERR_UNSUPPORTED
    assert fused(mu=0) == tc.TC_OK

    def expand(**k):
        return lib.tc_embed_expand(k.get("g", h.fp()), k.get("nb", 10), k.get("dim", 8),
                                   k.get("bo", h.ip()), k.get("n", 10), k.get("e", h.fp()), None)
    assert expand(dim=2) == tc.TC_ERR_UNSUPPORTED
    assert expand(n=-1) == tc.TC_ERR_INVALID_ARG
    assert expand(e=None) == tc.TC_ERR_INVALID_ARG
    assert expand(e=h.fp(misalign=True)) == tc.TC_ERR_UNSUPPORTED
    assert expand(n=0) == tc.TC_OK

    def coalesce(**k):
        return lib.tc_embed_coalesce(k.get("e", h.fp()), k.get("n", 10), k.get("dim", 8),
                                     k.get("so", h.ip()), k.get("sp", h.ip()), k.get("nu", h.ip()),
                                     k.get("mu", 10), k.get("coal", h.fp()), k.get("ws", None),
                                     k.get("wsb", 0), None)
    assert coalesce(dim=1030) == tc.TC_ERR_UNSUPPORTED
    assert coalesce(wsb=64) == tc.TC_ERR_INVALID_ARG
    assert coalesce(mu=-3) == tc.TC_ERR_INVALID_ARG
    assert coalesce(sp=None) == tc.TC_ERR_INVALID_ARG
    assert coalesce(mu=0) == tc.TC_OK
    assert h.untouched()


def test_noalloc_backward_update_rejects_bad_arguments(tc):
    """The no-allocation variant: the checks of tc_embed_backward_update,
    plus its scratch limit, all before anything is launched or looked up."""
    lib, h = tc._lib, HostBuffers()

    def f(**k):
        return lib.tc_embed_backward_update_noalloc(
            k.get("g", h.fp()), k.get("nb", 10), k.get("dim", 8), k.get("so", h.ip()),
            k.get("cs", h.ip()), k.get("ur", h.ip()), k.get("nu", h.ip()), k.get("mu", 10),
            k.get("n", 100), k.get("W", h.fp()), k.get("A", None), k.get("rows", 100),
            k.get("opt", 0), 0.01, 1e-8, k.get("gamma", 0.9), k.get("coal", None), None)
    assert f(dim=6) == tc.TC_ERR_UNSUPPORTED and "noalloc" in _err(tc)
    assert f(opt=3, A=h.fp()) == tc.TC_ERR_UNSUPPORTED
    assert f(opt=1) == tc.TC_ERR_INVALID_ARG
    assert f(W=None) == tc.TC_ERR_INVALID_ARG
    assert f(n=-1) == tc.TC_ERR_INVALID_ARG
    assert f(n=2 ** 31) == tc.TC_ERR_INVALID_ARG
    over = 40_000_000
    assert tc.tc_backward_workspace_bytes(over, 64) > tc.TC_NOALLOC_SCRATCH_BYTES
    assert f(n=over, dim=64) == tc.TC_ERR_WORKSPACE and "scratch" in _err(tc)
    assert f(n=over, dim=64, mu=0) == tc.TC_ERR_WORKSPACE
    assert f(mu=0) == tc.TC_OK and _err(tc) == ""     # nothing to do, nothing looked up
    assert h.untouched()


def test_forward_cast_rejects_bad_arguments(tc):
    lib, h = tc._lib, HostBuffers()
    need = lib.tc_cast_workspace_bytes(1000, 100, 1)

    def f(**k):
        return lib.tc_embed_forward_cast(
            k.get("W", h.fp()), k.get("rows", 100), k.get("dim", 64), k.get("off", h.lp()),
            k.get("T", 1), k.get("B", 50), k.get("mtr", 100), k.get("idx", h.ip()),
            k.get("bo", h.ip()), k.get("n", 1000), k.get("out", h.fp()), k.get("ur", h.ip()),
            k.get("so", h.ip()), k.get("cs", h.ip()), None, k.get("nu", h.ip()),
            k.get("ws", h.wsp()), k.get("wsb", need), None)
    assert f(dim=6) == tc.TC_ERR_UNSUPPORTED and "tc_embed_forward_cast" in _err(tc)
    assert f(dim=2048) == tc.TC_ERR_UNSUPPORTED
    assert f(W=None) == tc.TC_ERR_INVALID_ARG and "null" in _err(tc)
    assert f(out=None) == tc.TC_ERR_INVALID_ARG
    assert f(out=h.fp(misalign=True)) == tc.TC_ERR_UNSUPPORTED
    assert f(T=-1) == tc.TC_ERR_INVALID_ARG
    # the cast's own checks, before the forward is launched
    assert f(wsb=need - 1) == tc.TC_ERR_WORKSPACE
    assert f(n=2 ** 31) == tc.TC_ERR_INVALID_ARG
    assert f(rows=2 ** 31) == tc.TC_ERR_INVALID_ARG
    assert f(cs=None) == tc.TC_ERR_INVALID_ARG
    assert f(mtr=-1) == tc.TC_ERR_INVALID_ARG
    assert h.untouched()


def test_check_index_rejects_bad_arguments(tc):
    lib, h = tc._lib, HostBuffers()

    def f(**k):
        return lib.tc_check_index(k.get("off", h.lp()), k.get("T", 1), k.get("B", 50),
                                  k.get("rows", 100), k.get("mtr", 0), k.get("idx", h.ip()),
                                  k.get("bo", h.ip()), k.get("n", 1000), k.get("rep", h.lp()),
                                  None)
    assert f(rep=None) == tc.TC_ERR_INVALID_ARG and "null" in _err(tc)
    assert f(rep=h.lp() + 4) == tc.TC_ERR_INVALID_ARG and "aligned" in _err(tc)
    assert f(off=None) == tc.TC_ERR_INVALID_ARG
    assert f(bo=None) == tc.TC_ERR_INVALID_ARG
    assert f(idx=None) == tc.TC_ERR_INVALID_ARG
    assert f(T=-1) == tc.TC_ERR_INVALID_ARG and "negative" in _err(tc)
    assert f(mtr=-1) == tc.TC_ERR_INVALID_ARG
    assert f(n=2 ** 31) == tc.TC_ERR_INVALID_ARG
    assert f(rows=2 ** 31) == tc.TC_ERR_INVALID_ARG
    assert f(T=2 ** 16, B=2 ** 15) == tc.TC_ERR_INVALID_ARG and "bags" in _err(tc)
    assert h.untouched()


def test_launch_without_device_reports_hip_error(tc):
    """With valid arguments but no GPU, the launch fails and is reported as
    TC_ERR_HIP with the runtime's message (the kernel never runs)."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present; this checks the no-device path only")
    lib, h = tc._lib, HostBuffers()
    st = lib.tc_embed_forward(h.fp(), 100, 8, h.lp(), 1, 4, h.ip(), h.ip(), h.fp(), None)
    assert st == tc.TC_ERR_HIP
    assert "k_forward" in _err(tc)
    assert h.untouched()
