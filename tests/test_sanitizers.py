"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only): the oracle (clang, -fsanitize=address,undefined) and libtc's host
side (argument checks, workspace layout, error paths; the GPU code is built
as usual) are rebuilt with the sanitizers, and the host-side tests that
exercise them run in a child process that preloads clang's sanitizer
runtime. Any report fails the child (halt_on_error)."""
import glob
import os
import subprocess
import sys

import pytest

import oracle
from paper_2010_13100_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RUNTIME = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))


@pytest.mark.skipif(not RUNTIME, reason="clang's AddressSanitizer runtime is not installed")
def test_host_code_under_sanitizers():
    oracle.build(san=True)
    B.build(sanitize=True)
    env = dict(os.environ, TC_SANITIZED="1", LD_PRELOAD=RUNTIME[-1],
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    files = ["tests/test_abi.py", "tests/test_oracle_pins.py", "tests/test_summation_order.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider", *files], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=900)
    print(r.stdout[-3000:], r.stderr[-3000:])
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout and "AddressSanitizer" not in r.stderr
    assert "runtime error" not in r.stderr
