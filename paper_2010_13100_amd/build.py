"""Compile the HIP libraries of the package for gfx950 (in-tree).

  libtc.so           the training-step library (include/tc.h)
  libtc_workload.so  device-side fill of synthetic tables (include/tc_workload.h)

Flags: -O3; -ffp-contract=off so no multiply-add is fused (the arithmetic is
separately rounded fp32 everywhere); packed-fp32 instructions are disabled.
Each source is compiled to an object of its own (in parallel, under
_build/), then linked.

sanitize=True builds libtc_san.so instead: the same sources with
AddressSanitizer and UndefinedBehaviorSanitizer on the host code only (the
GPU code is built as usual), for running the host-side tests under the
sanitizers (tests/test_sanitizers.py).
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
         f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-I" + INCLUDE, "-I" + CSRC]
# host code only: each -fsanitize= right after -Xarch_host
SAN_FLAGS = ["-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
             "-fno-omit-frame-pointer"]

LIBS = {
    "libtc.so": ["tc_api.hip", "tc_gather_reduce.hip", "tc_backward.hip", "tc_cast.hip",
                 "tc_update.hip", "tc_check.hip"],
    "libtc_workload.so": ["workload_fill.hip"],
}


def lib_path(name: str) -> str:
    return os.path.join(PKG, name)


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed: {' '.join(cmd[-3:])}")


def build_lib(name: str, sources, out: str, extra=(), verbose=False, tag="") -> None:
    os.makedirs(BUILD, exist_ok=True)
    objs = [os.path.join(BUILD, os.path.splitext(s)[0] + tag + ".o") for s in sources]
    cmds = [[HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, s), "-o", o]
            for s, o in zip(sources, objs)]
    with ThreadPoolExecutor(max_workers=min(8, len(cmds))) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = out + ".tmp"
    # a sanitized library is linked without its runtime: the process that
    # loads it preloads the sanitizer runtime, which defines those symbols
    _run([HIPCC, *FLAGS, "-shared", *objs, "-o", tmp], verbose)
    os.replace(tmp, out)


def build(verbose: bool = False, sanitize: bool = False) -> None:
    if sanitize:
        build_lib("libtc.so", LIBS["libtc.so"], lib_path("libtc_san.so"), SAN_FLAGS, verbose,
                  tag=".san")
        return
    for name, sources in LIBS.items():
        build_lib(name, sources, lib_path(name), (), verbose)


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv)
