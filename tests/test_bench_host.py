"""Host logic of bench.py and the workload variants (no GPU)."""
import os
import subprocess
import sys

import bench
from paper_2010_13100_amd import workload as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_algorithmic_bytes_per_optimizer():
    n, u, nb = 1000, 300, 40
    base = wl.WORKLOADS["c2"]
    D4 = 4 * base.dim
    got = {o: bench.algorithmic_bytes(wl.variant(base, optimizer=o), n, u, nb)
           for o in ("sgd", "adagrad", "rmsprop", "rowwise_adagrad")}
    assert got["sgd"]["update"] == u * 4 + 3 * u * D4
    assert got["adagrad"]["update"] == got["rmsprop"]["update"] == u * 4 + 5 * u * D4
    assert got["rowwise_adagrad"]["update"] == u * 4 + 3 * u * D4 + 8 * u
    # fused: no coalesced row written or read back
    assert got["sgd"]["backward_update"] == (got["sgd"]["backward"] + got["sgd"]["update"]
                                             - 2 * u * D4)
    assert got["sgd"]["forward"] == n * 4 + (nb + 1) * 4 + n * D4 + nb * D4


def test_variant_names_and_identity():
    w = wl.WORKLOADS["c3"]
    assert wl.variant(w) is w
    assert wl.variant(w, batch=w.batch, dim=w.dim, optimizer=w.optimizer) is w
    v = wl.variant(w, batch=1024, dim=32, optimizer="rmsprop")
    assert v.name == "8x5M-d32-b1024-poisson40-zipf1.2-rmsprop"
    assert (v.batch, v.dim, v.optimizer, v.cfg_id) == (1024, 32, "rmsprop", w.cfg_id)


def _run(*a):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *a],
                          capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_step_calls_per_flag():
    """The calls one timed step makes: forward and cast in one call unless
    --no-overlap or --unfused, backward and update in one pass unless
    --unfused or the optimizer is row-wise Adagrad."""
    import argparse
    ns = lambda **k: argparse.Namespace(**{"unfused": False, "no_overlap": False, **k})  # noqa
    c2 = wl.WORKLOADS["c2"]
    rw = wl.variant(c2, optimizer="rowwise_adagrad")
    assert bench.step_calls(ns(), c2) == ["forward_cast", "backward_update"]
    assert bench.step_calls(ns(no_overlap=True), c2) == ["forward", "cast", "backward_update"]
    assert bench.step_calls(ns(unfused=True), c2) == ["forward", "cast", "backward", "update"]
    assert bench.step_calls(ns(), rw) == ["forward_cast", "backward", "update"]
    # every call has its algorithmic bytes, kernels and sources
    b = bench.algorithmic_bytes(c2, 1000, 300, 40)
    for c in ("forward_cast", "forward", "cast", "backward_update", "backward", "update"):
        assert c in b and c in bench.KERNEL_NAMES and c in bench.KERNEL_SOURCES
    assert b["forward_cast"] == b["forward"] + b["cast"]
