"""Compile the HIP libraries of the package for gfx950 (in-tree).

  libtc.so           the training-step library (include/tc.h)
  libtc_workload.so  device-side fill of synthetic tables (include/tc_workload.h)

Flags: -O3; -ffp-contract=off so no multiply-add is fused (the arithmetic is
separately rounded fp32 everywhere); packed-fp32 instructions are disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off",
         f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-I" + INCLUDE, "-I" + CSRC]

LIBS = {
    "libtc.so": ["tc_api.hip", "tc_gather_reduce.hip", "tc_backward.hip", "tc_cast.hip",
                 "tc_update.hip", "tc_check.hip"],
    "libtc_workload.so": ["workload_fill.hip"],
}


def lib_path(name: str) -> str:
    return os.path.join(PKG, name)


def build(verbose: bool = False) -> None:
    for name, sources in LIBS.items():
        out = lib_path(name)
        tmp = out + ".tmp"
        cmd = [HIPCC, *FLAGS, *[os.path.join(CSRC, s) for s in sources], "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            sys.stderr.write(r.stdout + r.stderr)
            raise RuntimeError(f"hipcc failed building {name}")
        os.replace(tmp, out)


if __name__ == "__main__":
    build(verbose=True)
