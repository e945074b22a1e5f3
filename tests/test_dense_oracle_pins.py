"""Pins for the dense continuous-input projection in the CPU oracle (no GPU).

y_m = s_m * sum_k Q_{m,k} x_k over row-major INT8 Q (paper Sec. 2.3, last
sentences; Fig. "execution", lower path), in float64.  Checked against
facts that do not come from the oracle: a hand-worked example (tests/golden),
numpy's int64 matrix product where x holds small integers (every step exact),
the x = e_k and all-ones special cases, linearity over dyadic inputs, row
permutations, and planted mistakes in a copy of the oracle source.
"""
import ctypes
import os
import subprocess
import sys

import numpy as np
import pytest

from tests.golden.load import load_dense_example

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def problem(M, K, B, seed, integer_x=False):
    rng = np.random.default_rng([42, 11, M, K, B, seed])
    Q = rng.integers(-127, 127, size=(M, K), dtype=np.int8, endpoint=True)
    s = rng.uniform(1e-3, 1e-2, M).astype(np.float32)
    if integer_x:
        x = rng.integers(-8, 8, size=(B, K), endpoint=True).astype(np.float32)
    else:
        x = rng.standard_normal((B, K)).astype(np.float32)
    return Q, s, x


def test_hand_worked_example(oracle_lib):
    g = load_dense_example()
    np.testing.assert_array_equal(oracle_lib.dense_forward(g["Q"], g["scale"], g["x"]), g["y"])


@pytest.mark.parametrize("M,K", [(1, 1), (3, 7), (16, 64), (33, 100), (64, 1536)])
@pytest.mark.parametrize("B", [1, 3])
def test_integer_inputs_match_int64_product(oracle_lib, M, K, B):
    """With integer x every product and partial sum is an integer below
    2^53, so the float64 oracle must equal numpy's int64 matmul times the
    scale exactly (the scale times an integer below 2^24 is exact too)."""
    Q, s, x = problem(M, K, B, seed=1, integer_x=True)
    dot = x.astype(np.int64) @ Q.astype(np.int64).T
    np.testing.assert_array_equal(oracle_lib.dense_forward(Q, s, x), dot.astype(np.float64) * s.astype(np.float64))


def test_unit_vectors_select_a_column(oracle_lib):
    Q, s, _ = problem(20, 37, 1, seed=2)
    for k in (0, 5, 36):
        e = np.zeros((1, 37), np.float32)
        e[0, k] = 1.0
        np.testing.assert_array_equal(oracle_lib.dense_forward(Q, s, e)[0], Q[:, k].astype(np.float64) * s)


def test_all_ones_gives_scaled_row_sums(oracle_lib):
    Q, s, _ = problem(20, 300, 1, seed=3)
    y = oracle_lib.dense_forward(Q, s, np.ones((1, 300), np.float32))[0]
    np.testing.assert_array_equal(y, Q.astype(np.int64).sum(axis=1).astype(np.float64) * s)


def test_linearity_on_dyadic_inputs(oracle_lib):
    """x1 + 2 * x2 with x on a 1/8 grid: all sums exact, so y is exactly linear."""
    rng = np.random.default_rng(4)
    Q, s, _ = problem(10, 50, 1, seed=4)
    x1 = (rng.integers(-64, 64, (1, 50)) / 8).astype(np.float32)
    x2 = (rng.integers(-64, 64, (1, 50)) / 8).astype(np.float32)
    y = lambda x: oracle_lib.dense_forward(Q, s, x)
    np.testing.assert_array_equal(y(x1 + 2 * x2), y(x1) + 2 * y(x2))


def test_row_permutation_and_zero_rows(oracle_lib):
    Q, s, x = problem(12, 40, 2, seed=5)
    Q[3] = 0
    perm = np.random.default_rng(6).permutation(12)
    y = oracle_lib.dense_forward(Q, s, x)
    np.testing.assert_array_equal(oracle_lib.dense_forward(Q[perm], s[perm], x), y[:, perm])
    assert (y[:, 3] == 0).all()


def test_general_inputs_close_to_a_correctly_rounded_sum(oracle_lib):
    """Real-valued x: the oracle's float64 sum agrees with math.fsum (exactly
    rounded) to within its own K * 2^-53 bound."""
    import math
    Q, s, x = problem(8, 1000, 2, seed=7)
    y = oracle_lib.dense_forward(Q, s, x)
    for b in range(2):
        for m in range(8):
            terms = [float(Q[m, k]) * float(x[b, k]) for k in range(1000)]
            exact = math.fsum(terms) * float(s[m])
            bound = 1000 * 2.0 ** -53 * sum(abs(t) for t in terms) * float(s[m]) + 2.0 ** -52 * abs(exact)
            assert abs(y[b, m] - exact) <= bound


MUTATIONS = {
    "column-major read": ("const int8_t *row = Q + m * K;", "const int8_t *row = Q + m;"),
    "dropped last input": ("for (int64_t k = 0; k < K; ++k)\n                dot +=", "for (int64_t k = 0; k + 1 < K; ++k)\n                dot +="),
    "scale of the wrong row": ("y[b * M + m] = (double)scale[m] * dot;", "y[b * M + m] = (double)scale[(m + 1) % M] * dot;"),
    "unsigned weights": ("dot += (double)row[k] * (double)xb[k];", "dot += (double)(uint8_t)row[k] * (double)xb[k];"),
    "activation of the wrong batch row": ("const float *xb = x + b * K;", "const float *xb = x;"),
}


def _pins_pass(lib):
    ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    lib.oracle_dense_forward.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    g = load_dense_example()
    Q, s, x = problem(9, 33, 2, seed=8, integer_x=True)
    cases = [(g["Q"], g["scale"], g["x"], g["y"]),
             (Q, s, x, (x.astype(np.int64) @ Q.astype(np.int64).T).astype(np.float64) * s.astype(np.float64))]
    for Q, s, x, ref in cases:
        M, K = Q.shape
        y = np.zeros((x.shape[0], M), np.float64)
        lib.oracle_dense_forward(ptr(np.ascontiguousarray(Q)), ptr(s), K, M, ptr(np.ascontiguousarray(x)), x.shape[0], ptr(y))
        if not np.array_equal(y, ref):
            return False
    return True


def _build(tmp_path, old, new):
    src = open(os.path.join(ROOT, "oracle", "spike_oracle.c")).read()
    assert src.count(old) == 1, f"mutation anchor missing or ambiguous: {old!r}"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-fPIC", "-shared", "-pthread", "-ffp-contract=off",
                    str(path), "-o", str(lib)], check=True)
    return lib


def _pins_pass_isolated(lib_path):
    code = ("import sys, ctypes; sys.path.insert(0, %r); "
            "from tests.test_dense_oracle_pins import _pins_pass; "
            "sys.exit(0 if _pins_pass(ctypes.CDLL(%r)) else 1)") % (ROOT, str(lib_path))
    return subprocess.run([sys.executable, "-c", code], capture_output=True).returncode == 0


def test_unmutated_copy_passes_pins(tmp_path):
    assert _pins_pass_isolated(_build(tmp_path, "#include <stdint.h>", "#include <stdint.h>"))


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(tmp_path, name):
    old, new = MUTATIONS[name]
    assert not _pins_pass_isolated(_build(tmp_path, old, new)), f"pins missed mutation: {name}"
