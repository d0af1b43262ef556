"""Planted mistakes in a copy of the oracle source must trip at least one pin.

Each case rewrites one line of ``oracle/tc_oracle.c`` into a plausible bug (a
dropped term, a wrong sign or index, a lost tie-break, a transposed operand),
builds the copy with gcc into a temporary directory, and runs every pin
against it. The shipped oracle is never modified.
"""
import json
import os
import subprocess
import sys

import pytest

import oracle
from paper_2010_13100_amd import workload as wl
from tests import pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "tc_oracle.c")

MUTATIONS = {
    # forward keeps only the last gathered row instead of summing
    "forward_no_accumulate": ("o[d] = o[d] + w[d];", "o[d] = w[d];"),
    # Algorithm 1 without carrying prev forward: nothing is coalesced
    "coalesce_no_prev_update": ("        prev = curr;\n", "\n"),
    # Algorithm 1 drops the first gradient of every segment
    "coalesce_drop_first": ("memcpy(coal + i * dim, e, sizeof(real) * (size_t)dim);",
                            "memset(coal + i * dim, 0, sizeof(real) * (size_t)dim);"),
    # unstable sort: ties in reverse input order
    "sort_ties_reversed": ("return x->pos < y->pos ? -1 : 1;", "return x->pos < y->pos ? 1 : -1;"),
    # Algorithm 2 without the first flag
    "casting_scan0_zero": ("scan[0] = 1;", "scan[0] = 0;"),
    # Algorithm 2 takes sorted src instead of sorted dst as the casted src
    "casting_src_swapped": ("casted_src[i] = dst[sorted_pos[i]];",
                            "casted_src[i] = (int32_t)src[sorted_pos[i]];"),
    # Algorithm 3 with src and dst transposed
    "gather_reduce_transposed": (
        "real *c = coal + (int64_t)casted_dst[i] * dim;\n        const real *g = grad_out + (int64_t)casted_src[i] * dim;",
        "real *c = coal + (int64_t)casted_src[i] * dim;\n        const real *g = grad_out + (int64_t)casted_dst[i] * dim;"),
    # SGD with the sign flipped
    "sgd_sign": ("w[d] = w[d] - t;", "w[d] = w[d] + t;"),
    # Adagrad without epsilon
    "adagrad_no_eps": ("a[d] = a[d] + sq;\n            real s = real_sqrt(reps + a[d]);",
                       "a[d] = a[d] + sq;\n            real s = real_sqrt(a[d]);"),
    # Adagrad dividing by the accumulator before it is updated
    "adagrad_stale_acc": ("a[d] = a[d] + sq;\n            real s = real_sqrt(reps + a[d]);",
                          "real s = real_sqrt(reps + a[d]);\n            a[d] = a[d] + sq;"),
    # RMSprop with gamma and 1 - gamma swapped
    "rmsprop_gamma_swapped": ("real t = rg * a[d];", "real t = rc * a[d];"),
    # RMSprop without the (1 - gamma) factor on the new squared gradient
    "rmsprop_no_one_minus_gamma": ("real m = rc * sq;", "real m = sq;"),
    # RMSprop dividing by sqrt(A) without epsilon
    "rmsprop_no_eps": ("a[d] = t + m;\n            real s = real_sqrt(reps + a[d]);",
                       "a[d] = t + m;\n            real s = real_sqrt(a[d]);"),
    # row-wise Adagrad adding the row's sum of squares instead of its mean
    "rowwise_sum_not_mean": ("real m = ss / rdim;", "real m = ss;"),
    # row-wise Adagrad squaring only the first column
    "rowwise_first_column": ("real sq = g[d] * g[d];\n            ss = ss + sq;",
                             "real sq = g[0] * g[0];\n            ss = ss + sq;"),
    # row-wise Adagrad not keeping its accumulator across steps
    "rowwise_acc_reset": ("a[0] = a[0] + m;", "a[0] = m;"),
    # expand reads the gradient of the wrong bag (off by one)
    "expand_off_by_one": ("grad_out + (int64_t)dst[j] * dim", "grad_out + (int64_t)(dst[j] > 0 ? dst[j] - 1 : 0) * dim"),
    # pairs from CSR forget the table's row offset
    "pairs_no_table_offset": ("src[j] = table_row_offset[t] + indices[j];", "src[j] = indices[j];"),
}


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# A mutant can write out of bounds, so it runs in a child process; a crash of
# that process counts as caught, like a failed pin.
_CHILD = """
import json, sys
sys.path.insert(0, {root!r})
import oracle
from tests import pins
orc = oracle.Oracle("f64", path={lib!r})
failed = []
for pin in pins.ALL_PINS:
    try:
        pin(orc)
    except (AssertionError, oracle.OracleError):
        failed.append(pin.__name__)
print(json.dumps(failed))
"""


def _pins_fail(lib: str) -> list:
    r = subprocess.run([sys.executable, "-c", _CHILD.format(root=ROOT, lib=lib)],
                       capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        return [f"crashed (exit {r.returncode})"]
    return json.loads(r.stdout.strip().splitlines()[-1])


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, tmp_path):
    old, new = MUTATIONS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation anchor for {name} not unique"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(text.replace(old, new))
    lib = tmp_path / "libmutant.so"
    oracle.build_one(str(mutated), "f64", str(lib))
    failed = _pins_fail(str(lib))
    assert failed, f"no pin caught mutation {name}"


def test_rounding_bound_catches_f32_mistake(tmp_path):
    """A planted fp32-only mistake (a sum that skips every 8th term) is caught by
    the f32-against-f64 bound even where it keeps most of each sum."""
    text = open(SRC).read()
    old = "c[d] = c[d] + e[d];"
    assert text.count(old) == 1
    mutated = tmp_path / "mutant.c"
    mutated.write_text(text.replace(old, "if ((j & 7) != 7) c[d] = c[d] + e[d];"))
    lib = tmp_path / "libmutant32.so"
    oracle.build_one(str(mutated), "f32", str(lib))
    w = wl.WORKLOADS["c2"].scaled(name="c2-tiny", num_tables=2, rows_per_table=2000, batch=64)
    b = wl.make_batch(w, step=2)
    with pytest.raises(AssertionError):
        pins.check_f32_against_f64(oracle.Oracle("f32", path=str(lib)), oracle.Oracle("f64"), w, b)
