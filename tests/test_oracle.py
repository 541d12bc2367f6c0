"""The CPU oracle against its pins, and the pins against planted mistakes.

Every pin in oracle_pins.py runs against the real oracle (must pass).  Then
each entry of MUTANTS plants one plausible mistake into a copy of oracle.c
(wrong sign, dropped term, wrong or transposed index, wrong rounding, wrong
layout field), builds it with gcc, and requires at least one pin to fail.
Every mutant keeps all memory accesses in bounds.
"""
from __future__ import annotations

import os
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
import oracle_pins as P

ORACLE_C = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


# (name, original text, replacement, expected number of occurrences)
MUTANTS = [
    ("gemm_sign_flip",
     "(double)((int)q[k * N + n] - (int)z[gi * N + n])",
     "(double)((int)z[gi * N + n] - (int)q[k * N + n])", 1),
    ("gemm_drop_zero_point", "- (int)z[gi * N + n])", "- 0)", 1),
    ("gemm_drop_scale", "oracle_f16_to_f64(s[gi * N + n]);\n                }",
     "1.0;\n                }", 1),
    ("gemm_reversed_group_index",
     "int64_t gi = k / group;\n                    wcol",
     "int64_t gi = (K - 1 - k) / group;\n                    wcol", 1),
    ("gemm_transposed_x", "acc += xr[k] * wcol[k];", "acc += xd[k * M + m] * wcol[k];", 1),
    ("gemm_short_k_loop", "for (int64_t k = 0; k < K; ++k)\n                        acc",
     "for (int64_t k = 0; k < K - 1; ++k)\n                        acc", 1),
    ("gemm_wrong_q_column", "(int)q[k * N + n]", "(int)q[k * N + (N - 1 - n)]", 1),
    ("gemm_wrong_s_column", "oracle_f16_to_f64(s[gi * N + n]);\n                }",
     "oracle_f16_to_f64(s[gi * N + (n ^ 1)]);\n                }", 1),
    ("dequant_sign_flip", "(double)(qv - zv)", "(double)(zv - qv)", 1),
    ("dequant_group_as_row", "int64_t gi = k / group;\n        for",
     "int64_t gi = (k / group + 1) % (K / group);\n        for", 1),
    ("f16_exponent_bias", "e - 25", "e - 24", 1),
    ("f16_subnormal_scale", "ldexp((double)f, -24)", "ldexp((double)f, -23)", 1),
    ("f16_round_ties_away", "rint(ldexp(a, 10 - ex))", "round(ldexp(a, 10 - ex))", 1),
    ("f16_no_subnormal_clamp", "if (ex < -14)\n        ex = -14;", "if (ex < -24)\n        ex = -24;", 1),
    ("pack_slot_identity", "(int)(e / 2 + 4 * (e % 2))", "(int)e", 1),
    ("pack_lane_group_reversed", "int64_t lane = 16 * g + c;", "int64_t lane = 16 * (3 - g) + c;", 1),
    ("pack_swap_step_and_group", "int64_t j = r / 32, g = (r % 32) / 8,",
     "int64_t g = r / 32, j = (r % 32) / 8,", 1),
    ("pack_zero_nibble_reversed", "v << (4 * (c % 8))", "v << (4 * (7 - c % 8))", 1),
    ("pack_scale_reversed", "ps[(nt * KG + kg) * 16 + c]", "ps[(nt * KG + kg) * 16 + (15 - c)]", 1),
]


def _run_pins():
    failed = []
    for pin in P.ALL_PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
    return failed


@pytest.fixture(scope="module")
def oracle_source():
    with open(ORACLE_C) as f:
        return f.read()


@pytest.mark.parametrize("name,old,new,count", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(oracle_source, name, old, new, count):
    assert oracle_source.count(old) == count, "mutation site for %s not found" % name
    src = oracle_source.replace(old, new)
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "mut.c")
        so = os.path.join(d, "libmut.so")
        with open(c, "w") as f:
            f.write(src)
        subprocess.run(["gcc", "-O1", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-o", so, c, "-lm"],
                       check=True)
        with oracle.use_library(so):
            failed = _run_pins()
    assert failed, "no pin caught the planted mistake %s" % name


def test_oracle_error_paths():
    q = np.zeros((256, 16), np.uint8)
    z = np.zeros((2, 16), np.uint8)
    s = np.zeros((2, 16), np.uint16)
    q[3, 4] = 16
    with pytest.raises(oracle.OracleError):
        oracle.gemm(np.zeros((1, 256), np.uint16), q, z, s)
    with pytest.raises(oracle.OracleError):
        oracle.pack(q, z, s)
    q[3, 4] = 0
    with pytest.raises(oracle.OracleError):
        oracle.pack(q, z, s, group=64)
    # M = 0 is a valid, empty GEMM
    assert oracle.gemm(np.zeros((0, 256), np.uint16), q, z, s).shape == (0, 16)
