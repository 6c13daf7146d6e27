"""The oracle's pins catch plausible mistakes in the oracle itself.

Each case builds a copy of ``oracle/gett_oracle.c`` with one planted mistake
(on the CPU, with gcc), routes the oracle through it and runs a selection of
the pins of ``test_oracle_pins.py``: at least one of them must fail.  The
mistakes are the kinds a reader could make when writing Eq. 3 and the parity
metric's denominator from the paper: a signed instead of an absolute factor in
den64, a dropped |beta||c| term, a product dropped from the sum, a wrong sign
on beta * C, the free indices of A and B exchanged (a transposed operand).
"""
import os
import subprocess

import numpy as np
import pytest

import oracle
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "gett_oracle.c")

# (name, text in the source, replacement)
MUTANTS = [
    ("den: alpha instead of |alpha|", "double d = fabs(alpha) * acc_abs;",
     "double d = alpha * acc_abs;"),
    ("den: a * b instead of |a||b|", "acc_abs += fabs(a) * fabs(b);", "acc_abs += a * b;"),
    ("den: |a| only", "acc_abs += fabs(a) * fabs(b);", "acc_abs += fabs(a);"),
    ("den: |beta||c| dropped", "d += fabs(beta) * fabs(c);", "d += 0.0;"),
    ("den: beta instead of |beta|", "d += fabs(beta) * fabs(c);", "d += beta * fabs(c);"),
    ("den: |alpha| applied twice", "double d = fabs(alpha) * acc_abs;",
     "double d = fabs(alpha) * fabs(alpha) * acc_abs;"),
    ("out: first product dropped", "acc += a * b;", "if (y > 0) acc += a * b;"),
    ("out: beta * C subtracted", "r += beta * c;", "r -= beta * c;"),
    ("out: free strides of A and B exchanged",
     "offA += idx * P->strA_of_c[i];\n        offB += idx * P->strB_of_c[i];",
     "offA += idx * P->strB_of_c[i];\n        offB += idx * P->strA_of_c[i];"),
]


def pin_suite():
    """(name, callable) pairs: pins run with fixed parameters."""
    return [
        ("den hand 2x2x2", pins.test_den_hand_computed_2x2x2),
        *[(f"den unit {s}", lambda s=s: pins.test_den_of_unit_magnitudes_is_contracted_size(s))
          for s in range(6)],
        *[(f"den bounds {s}", lambda s=s: pins.test_den_bounds_the_result_and_ignores_signs(s))
          for s in range(2)],
        *[(f"brute force {s}", lambda s=s: pins.test_brute_force_random_patterns(s))
          for s in range(1, 6)],
        ("all ones", pins.test_all_ones_gives_contracted_size),
        ("gemm by definition", lambda: pins.test_gemm_by_definition(5, 6, 7, 0.5)),
    ]


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("oracle_mutants")


def build_mutant(src_text, old, new, path):
    assert src_text.count(old) == 1, f"planted mistake not found once: {old!r}"
    c = path.with_suffix(".c")
    c.write_text(src_text.replace(old, new))
    so = str(path.with_suffix(".so"))
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-o", so,
                           str(c), "-lm"])
    return so


def test_unmutated_copy_passes_the_suite(mutant_dir):
    """The harness itself: a copy of the unchanged source passes every pin."""
    text = open(SRC).read()
    so = build_mutant(text, "double d = fabs(alpha) * acc_abs;",
                      "double d = fabs(alpha) * acc_abs;", mutant_dir / "same")
    with oracle.using_library(so):
        for name, fn in pin_suite():
            fn()


@pytest.mark.parametrize("case", range(len(MUTANTS)), ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(mutant_dir, case):
    name, old, new = MUTANTS[case]
    text = open(SRC).read()
    so = build_mutant(text, old, new, mutant_dir / f"m{case}")
    failed = []
    with oracle.using_library(so):
        for pname, fn in pin_suite():
            try:
                fn()
            except (AssertionError, ValueError):
                failed.append(pname)
    assert failed, f"no pin caught the planted mistake: {name}"
    # and the oracle in use afterwards is the real one again
    r = oracle.contract("m,n", "m,k", "k,n", np.ones((2, 3)), np.ones((3, 2)), -1.0, 0.0,
                        shape_C=[2, 2])
    assert np.all(r.den64 == 3.0)
