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


def test_compulsory_bytes_read_each_distinct_row_once():
    """The compulsory bound replaces the gathers of the paper's model (one
    row per pair) by one read per distinct row: the forward's U table rows
    and the backward's T*B output-gradient rows."""
    n, u, nb = 1000, 300, 40
    for o in ("sgd", "adagrad"):
        w = wl.variant(wl.WORKLOADS["c3"], optimizer=o)
        D4 = 4 * w.dim
        a, c = bench.algorithmic_bytes(w, n, u, nb), bench.compulsory_bytes(w, n, u, nb)
        assert a["forward"] - c["forward"] == (n - u) * D4
        assert a["backward"] - c["backward"] == (n - nb) * D4
        assert a["backward_update"] - c["backward_update"] == (n - nb) * D4
        assert c["forward_cast"] == c["forward"] + c["cast"] and c["cast"] == a["cast"]
        assert c["update"] == a["update"]


def test_traffic_from_counter_csvs(tmp_path, monkeypatch):
    """Counter CSVs of a --profile-steps run turn into bytes per call launch:
    every dispatch of a call's kernels, scaled by the copy calibration, over
    the number of steps."""
    import json

    def csv(sub, rows):
        d = tmp_path / sub
        d.mkdir()
        lines = ["Kernel_Name,Counter_Value"] + [f'"{k}",{v}' for k, v in rows]
        (d / "run_counter_collection.csv").write_text("\n".join(lines) + "\n")

    csv("copy_fetch", [("copyBuffer", 512.0)] * 2)        # KiB: half of a 1 MiB copy
    csv("copy_write", [("copyBuffer", 1024.0)] * 2)
    csv("fetch", [("void tc::k_forward_build<16>(x)", 100.0), ("k_radix_scatter<8>", 10.0),
                  ("k_radix_scatter<8>", 10.0), ("k_backward_short<16, 1>", 50.0),
                  ("k_backward_list", 5.0), ("fill_kernel", 999.0)] * 2)
    csv("write", [("void tc::k_forward_build<16>(x)", 1.0), ("k_radix_scatter<8>", 2.0),
                  ("k_radix_scatter<8>", 2.0), ("k_backward_short<16, 1>", 3.0),
                  ("k_backward_list", 4.0), ("fill_kernel", 999.0)] * 2)
    (tmp_path / "copy_bytes").write_text(str(1 << 20))
    (tmp_path / "steps").write_text("2")
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_sha", lambda call: "sha")
    t = bench.write_traffic(str(tmp_path), "cX", ["forward_cast", "backward_update"])
    fc, bu = t["forward_cast:cX"], t["backward_update:cX"]
    assert fc["fetch_bytes_per_launch"] == round((100 + 20) * 1024 * 2)
    assert fc["write_bytes_per_launch"] == round((1 + 4) * 1024)
    assert bu["fetch_bytes_per_launch"] == round(55 * 1024 * 2)
    assert bu["hbm_bytes_per_launch"] == bu["fetch_bytes_per_launch"] + 7 * 1024
    assert json.load(open(prof / "traffic.json"))["forward_cast:cX"] == fc


def test_host_cpu_reports_model_and_cores():
    h = bench.host_cpu()
    assert h["nproc"] >= 1 and isinstance(h["cpu_model"], str)
