"""Pins for the CPU oracle (runs without a GPU).

The oracle (oracle/spike_oracle.c) is the definition the GPU library is held
to, so it is itself checked here against facts that do not come from it:

* a hand-worked example derived on paper from Eq. (sparse) (tests/golden);
* numpy's int64 dense matrix-vector product over the unpacked 0/1 input,
  which is the product W x that the paper says the active-column sum equals
  (Sec. 1) -- an independent implementation of the definition;
* special cases: x = 0, x = 1 (row sums), x = e_k (column k), additivity
  over disjoint spike sets, complements, column permutations;
* the FP32 epilogue re-derived with numpy's IEEE binary32 multiply and as a
  correctly rounded float64 product;
* mutation checks: plausible mistakes planted in a copy of the oracle source
  are each caught by these pins.
"""
import ctypes
import os
import subprocess
import sys

import numpy as np
import pytest

from paper_2606_03026_amd import workloads as wl
from tests.golden.load import load_hand_example

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SHAPES = [1, 2, 7, 31, 32, 33, 63, 64, 65, 127, 200]


def dense_reference(W, bits):
    """W x over the unpacked 0/1 spikes, in int64 (numpy matmul)."""
    return bits.astype(np.int64) @ W.astype(np.int64)


def f32_bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def test_hand_worked_example(oracle_lib):
    g = load_hand_example()
    acc = oracle_lib.spike_acc(g["W"], g["masks"])
    np.testing.assert_array_equal(acc, g["acc"])
    out = oracle_lib.spike_forward(g["W"], g["scale"], g["masks"])
    np.testing.assert_array_equal(f32_bits(out), g["out_bits"])


def test_hand_example_active_lists(oracle_lib):
    g = load_hand_example()
    expect = [[0, 2, 3], [1, 4], [], [0, 1, 2, 3, 4]]
    for row, e in zip(g["masks"], expect):
        np.testing.assert_array_equal(oracle_lib.active_indices(row, g["K"]), e)


@pytest.mark.parametrize("K", SHAPES)
@pytest.mark.parametrize("N", [1, 7, 33, 64, 200])
@pytest.mark.parametrize("B", [0, 1, 3])
def test_matches_dense_integer_product(oracle_lib, K, N, B):
    p = wl.small_problem(K, N, B, p=0.37, seed=K * 1000 + N)
    acc = oracle_lib.spike_acc(p["W"], p["masks"])
    assert acc.shape == (B, N)
    np.testing.assert_array_equal(acc.astype(np.int64), dense_reference(p["W"], p["bits"]))


@pytest.mark.parametrize("K,N", [(1536, 1536), (6144, 1536), (200, 33)])
def test_special_cases(oracle_lib, K, N):
    rng = np.random.default_rng(K + N)
    W = rng.integers(-128, 127, size=(K, N), dtype=np.int8, endpoint=True)
    zero = np.zeros((1, K), bool)
    ones = np.ones((1, K), bool)
    # all-zero spikes: zero sums and +0.0 outputs
    acc0 = oracle_lib.spike_acc(W, wl.pack_bits(zero))
    assert not acc0.any()
    out0 = oracle_lib.spike_forward(W, np.full(N, 0.003, np.float32), wl.pack_bits(zero))
    assert not f32_bits(out0).any()
    # all-one spikes: row sums of Q
    np.testing.assert_array_equal(oracle_lib.spike_acc(W, wl.pack_bits(ones))[0],
                                  W.astype(np.int64).sum(axis=0))
    # one spike e_k: exactly column k
    for k in (0, K // 3, K - 1):
        e = np.zeros((1, K), bool)
        e[0, k] = True
        np.testing.assert_array_equal(oracle_lib.spike_acc(W, wl.pack_bits(e))[0], W[k].astype(np.int32))


def test_additive_over_disjoint_sets_and_complement(oracle_lib):
    K, N = 777, 130
    rng = np.random.default_rng(5)
    W = rng.integers(-128, 127, size=(K, N), dtype=np.int8, endpoint=True)
    x = rng.random(K) < 0.3
    y = (rng.random(K) < 0.3) & ~x
    acc = lambda bits: oracle_lib.spike_acc(W, wl.pack_bits(bits[None]))[0].astype(np.int64)
    np.testing.assert_array_equal(acc(x | y), acc(x) + acc(y))
    np.testing.assert_array_equal(acc(x) + acc(~x), W.astype(np.int64).sum(axis=0))


def test_column_permutation_invariance(oracle_lib):
    K, N = 300, 48
    rng = np.random.default_rng(6)
    W = rng.integers(-127, 127, size=(K, N), dtype=np.int8, endpoint=True)
    x = rng.random((2, K)) < 0.4
    perm = rng.permutation(K)
    a = oracle_lib.spike_acc(W, wl.pack_bits(x))
    b = oracle_lib.spike_acc(W[perm], wl.pack_bits(x[:, perm]))
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("K", [1, 63, 65, 100, 1535])
def test_padding_bits_ignored(oracle_lib, K):
    N = 9
    p = wl.small_problem(K, N, 2, 0.5, seed=3)
    junk = p["masks"].copy()
    valid = K % 64
    if valid:
        junk[:, -1] |= np.uint64(~((1 << valid) - 1) & 0xFFFFFFFFFFFFFFFF)
    np.testing.assert_array_equal(oracle_lib.spike_acc(p["W"], junk), oracle_lib.spike_acc(p["W"], p["masks"]))


def test_minus_128_weights(oracle_lib):
    K, N = 70, 5
    W = np.full((K, N), -128, np.int8)
    ones = np.ones((1, K), bool)
    np.testing.assert_array_equal(oracle_lib.spike_acc(W, wl.pack_bits(ones))[0], np.full(N, -128 * K))


def test_epilogue_is_one_binary32_multiply(oracle_lib):
    p = wl.small_problem(1536, 1536, 4, 0.1, seed=11)
    acc = oracle_lib.spike_acc(p["W"], p["masks"])
    out = oracle_lib.spike_forward(p["W"], p["scale"], p["masks"])
    # numpy's binary32 multiply (round to nearest even)
    np.testing.assert_array_equal(f32_bits(out), f32_bits(acc.astype(np.float32) * p["scale"]))
    # the float64 product of two binary32 numbers is exact, so rounding it
    # once to binary32 is the correctly rounded product
    exact = acc.astype(np.float64) * p["scale"].astype(np.float64)
    np.testing.assert_array_equal(f32_bits(out), f32_bits(exact.astype(np.float32)))


def test_subnormal_scale_not_flushed(oracle_lib):
    K, N = 3, 2
    W = np.array([[1, 1], [1, 1], [1, 1]], np.int8)
    scale = np.array([2.0 ** -140, 2.0 ** -149], np.float32)
    out = oracle_lib.spike_forward(W, scale, wl.pack_bits(np.ones((1, K), bool)))
    np.testing.assert_array_equal(f32_bits(out)[0], [0x600, 0x3])


@pytest.mark.parametrize("threads", [1, 2, 7, 64])
def test_thread_count_does_not_change_result(oracle_lib, threads):
    p = wl.small_problem(6144, 1536, 2, 0.1, seed=2)
    ref = oracle_lib.spike_forward(p["W"], p["scale"], p["masks"], threads=1)
    out = oracle_lib.spike_forward(p["W"], p["scale"], p["masks"], threads=threads)
    np.testing.assert_array_equal(f32_bits(out), f32_bits(ref))


def test_active_indices_match_flatnonzero(oracle_lib):
    for K in (1, 64, 65, 6144):
        bits = np.random.default_rng(K).random((1, K)) < 0.2
        np.testing.assert_array_equal(oracle_lib.active_indices(wl.pack_bits(bits)[0], K), np.flatnonzero(bits[0]))


def test_rejects_bad_arguments(oracle_lib):
    W = np.zeros((4, 3), np.int8)
    with pytest.raises(ValueError):
        oracle_lib.spike_forward(W, np.ones(4, np.float32), np.zeros((1, 1), np.uint64))  # scale length != N
    with pytest.raises(ValueError):
        oracle_lib.spike_acc(W, np.zeros((1, 2), np.uint64))  # wrong word count


# ---------------------------------------------------------------------------
# Mutation checks: each plausible mistake, planted in a copy of the oracle
# source, must make at least one of the pins above fail.
# ---------------------------------------------------------------------------

MUTATIONS = {
    "unsigned weights": ("acc[n - n0] += (int32_t)column[n];", "acc[n - n0] += (int32_t)(uint8_t)column[n];"),
    "dropped last active column": ("for (int64_t a = 0; a < n_active; ++a)", "for (int64_t a = 0; a + 1 < n_active; ++a)"),
    "transposed weight index": ("W + (int64_t)active[a] * N;", "W + (int64_t)active[a];"),
    "bit order reversed": ("(row[k / 64] >> (k % 64))", "(row[k / 64] >> (63 - k % 64))"),
    "padding bits counted": ("for (int64_t k = 0; k < K; ++k)", "for (int64_t k = 0; k < ((K + 63) / 64) * 64; ++k)"),
    "wrong sign": ("acc[n - n0] += (int32_t)column[n];", "acc[n - n0] -= (int32_t)column[n];"),
    "scale before sum": ("return as_float * scale;", "return (float)(as_float * (double)scale * 1.0000001);"),
    "scale index off": ("job->scale[n]", "job->scale[n - job->n0]"),
}


def _build_mutant(tmp_path, name, old, new):
    src = open(os.path.join(os.path.dirname(__file__), "..", "oracle", "spike_oracle.c")).read()
    assert src.count(old) >= 1, f"mutation anchor missing: {name}"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-fPIC", "-shared", "-pthread", "-ffp-contract=off",
                    str(path), "-o", str(lib)], check=True)
    return lib


def _pins_pass(lib):
    ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    lib.oracle_spike_acc.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                     ctypes.c_int64, ctypes.c_void_p]
    lib.oracle_spike_forward.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int]
    g = load_hand_example()
    cases = [(g["W"], g["scale"], g["masks"], g["acc"], g["out_bits"])]
    p = wl.small_problem(100, 37, 3, 0.4, seed=99)
    ref = dense_reference(p["W"], p["bits"]).astype(np.int32)
    cases.append((p["W"], p["scale"], p["masks"], ref, f32_bits(ref.astype(np.float32) * p["scale"])))
    for W, s, m, acc_ref, out_ref in cases:
        K, N = W.shape
        B = m.shape[0]
        acc = np.zeros((B, N), np.int32)
        lib.oracle_spike_acc(ptr(W), K, N, ptr(m), B, ptr(acc))
        if not np.array_equal(acc, acc_ref):
            return False
        for threads in (1, 3):
            out = np.zeros((B, N), np.float32)
            lib.oracle_spike_forward(ptr(W), ptr(s), K, N, ptr(m), B, ptr(out), threads)
            if not np.array_equal(f32_bits(out), out_ref):
                return False
    return True


def _pins_pass_isolated(lib_path):
    """Run the pins on a built copy in a child process: a mutant that writes
    out of bounds may crash, which also counts as caught."""
    code = ("import sys, ctypes; sys.path.insert(0, %r); "
            "from tests.test_oracle_pins import _pins_pass; "
            "sys.exit(0 if _pins_pass(ctypes.CDLL(%r)) else 1)") % (ROOT, str(lib_path))
    return subprocess.run([sys.executable, "-c", code], capture_output=True).returncode == 0


def test_unmutated_copy_passes_pins(tmp_path):
    _build_mutant(tmp_path, "none", "#include <stdint.h>", "#include <stdint.h>")
    assert _pins_pass_isolated(tmp_path / "libmutant.so")


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(tmp_path, name):
    old, new = MUTATIONS[name]
    _build_mutant(tmp_path, name, old, new)
    assert not _pins_pass_isolated(tmp_path / "libmutant.so"), f"pins missed mutation: {name}"
