"""Pins for the symmetric per-channel INT8 quantizer in the CPU oracle (no GPU).

s_m = max(max_k |W[m,k]|, 1e-8) / 127, Q = clip(round(W / s_m), -127, 127)
(paper Sec. 2.3), in binary32 with ties to even.  Checked against facts that
do not come from the oracle: a hand-worked fixture (tests/golden), the
reconstruction bound |Q s - W| <= s / 2, the row maximum landing on +-127,
sign symmetry, power-of-two scaling, permutation equivariance, a quotient
whose binary32 rounding creates a tie (which separates binary32 from exact
division), and planted mistakes in a copy of the oracle source.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import quant_oracle
from oracle.quant_oracle import export_column_major, quantize_int8
from tests.golden.load import load_quant_example

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def gaussian(M, K, seed, sigma=0.02):
    rng = np.random.default_rng([42, 12, M, K, seed])
    return rng.normal(0.0, sigma, size=(M, K)).astype(np.float32)


def check_hand_example(quantize):
    g = load_quant_example()
    Q, s = quantize(g["W"])
    np.testing.assert_array_equal(Q, g["Q"])
    for m, want in enumerate(g["scale"]):
        if want is not None:
            assert s[m] == np.float32(want), (m, s[m], want)
    floor = [m for m, w in enumerate(g["scale"]) if w is None]
    assert len({float(s[m]) for m in floor}) == 1 and s[floor[0]] > 0
    assert abs(float(s[floor[0]]) * 127 - 1e-8) < 1e-14


def check_reconstruction(quantize):
    W = gaussian(64, 300, 1)
    Q, s = quantize(W)
    err = np.abs(Q.astype(np.float64) * s[:, None].astype(np.float64) - W.astype(np.float64))
    assert (err <= s[:, None].astype(np.float64) * (0.5 + 2.0 ** -20)).all()


def check_row_max_maps_to_127(quantize):
    W = gaussian(50, 77, 2)
    W[3, 5] = -0.5  # the largest magnitude of row 3, negative
    Q, s = quantize(W)
    idx = np.argmax(np.abs(W), axis=1)
    np.testing.assert_array_equal(np.abs(Q[np.arange(50), idx]), 127)
    assert Q[3, 5] == -127
    assert (np.abs(Q) <= 127).all()


def check_binary32_tie(quantize):
    """x / s in binary32 is exactly n + 1/2 while the exact quotient lies just
    above it: binary32 arithmetic (ties to even) gives the even n; exact or
    float64 division would give n + 1."""
    for amax in (100.3, 139.1, 1.37, 201.9, 9.81):
        amax = np.float32(amax)
        s = np.float32(amax / np.float32(127))
        for n in range(0, 126, 2):
            x = np.float32(np.float64(n + 0.5) * np.float64(s))
            exact = Fraction(float(x)) / Fraction(float(s))
            if np.float32(x / s) == np.float32(n + 0.5) and exact > Fraction(2 * n + 1, 2):
                W = np.array([[amax, x, -x, 0]], dtype=np.float32)
                Q, sq = quantize(W)
                assert sq[0] == s
                assert (Q[0, 1], Q[0, 2]) == (n, -n), (float(amax), n, Q)
                break
        else:
            raise AssertionError(f"no tie case for amax {amax}")


CHECKS = [check_hand_example, check_reconstruction, check_row_max_maps_to_127, check_binary32_tie]


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_oracle_meets(check):
    check(quantize_int8)


def test_sign_symmetry_and_power_of_two_scaling():
    W = gaussian(40, 129, 3)
    Q, s = quantize_int8(W)
    Qn, sn = quantize_int8(-W)
    np.testing.assert_array_equal(Qn, -Q)
    np.testing.assert_array_equal(sn, s)
    for j in (-5, 3, 20):
        Qj, sj = quantize_int8((W * np.float32(2.0 ** j)).astype(np.float32))
        np.testing.assert_array_equal(Qj, Q)
        np.testing.assert_array_equal(sj, (s * np.float32(2.0 ** j)).astype(np.float32))


def test_permutations_commute():
    W = gaussian(30, 70, 4)
    Q, s = quantize_int8(W)
    rng = np.random.default_rng(5)
    pr, pc = rng.permutation(30), rng.permutation(70)
    Qp, sp = quantize_int8(np.ascontiguousarray(W[pr][:, pc]))
    np.testing.assert_array_equal(Qp, Q[pr][:, pc])
    np.testing.assert_array_equal(sp, s[pr])


def test_scales_are_per_output_channel_not_per_input():
    """Quantizing the transpose gives scales along the other axis (the export
    defect the paper withdraws): they differ from the per-output scales."""
    W = gaussian(6, 24, 6)
    W[:, 0] *= 8  # one large input column
    Q, s = quantize_int8(W)
    Qt, st = quantize_int8(np.ascontiguousarray(W.T))
    assert s.shape == (6,) and st.shape == (24,)
    assert not np.array_equal(Qt.T, Q)


def test_column_major_export_feeds_the_spike_oracle(oracle_lib):
    """W_cm[k, m] = Q[m, k]; the spike oracle on the export equals the int64
    brute force Q @ bits."""
    W = gaussian(48, 200, 7)
    Q, s = quantize_int8(W)
    Wcm = export_column_major(Q)
    assert Wcm.shape == (200, 48) and Wcm.flags.c_contiguous
    np.testing.assert_array_equal(Wcm.T, Q)
    rng = np.random.default_rng(8)
    bits = rng.random((3, 200)) < 0.3
    from paper_2606_03026_amd.workloads import pack_bits
    acc = oracle_lib.spike_acc(Wcm, pack_bits(bits))
    np.testing.assert_array_equal(acc, bits.astype(np.int64) @ Q.T.astype(np.int64))


def test_rejects_bad_input():
    with pytest.raises(ValueError):
        quantize_int8(np.zeros((3, 4), dtype=np.float64))
    with pytest.raises(ValueError):
        quantize_int8(np.zeros((0, 4), dtype=np.float32))
    with pytest.raises(ValueError):
        quantize_int8(np.zeros(4, dtype=np.float32))


MUTANTS = {
    "round half away from zero": ("np.rint(W[m] / s[m])",
                                  "np.sign(W[m] / s[m]) * np.floor(np.abs(W[m] / s[m]) + 0.5)"),
    "truncation": ("np.rint(W[m] / s[m])", "np.trunc(W[m] / s[m])"),
    "max over the input axis": ("np.max(np.abs(W[m]))", "np.max(np.abs(W[:, m % W.shape[1]]))"),
    "128 levels": ("QMAX = np.float32(127)", "QMAX = np.float32(128)"),
    "no floor": ("max(amax, FLOOR)", "amax"),
    "float64 division": ("np.rint(W[m] / s[m])", "np.rint(W[m].astype(np.float64) / np.float64(s[m]))"),
    "floor after the division": ("max(amax, FLOOR) / QMAX", "max(amax / QMAX, FLOOR)"),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistakes_are_caught(name):
    src = open(quant_oracle.__file__).read()
    old, new = MUTANTS[name]
    assert old in src
    ns = {}
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)
    failures = 0
    for check in CHECKS:
        try:
            with np.errstate(all="ignore"):
                check(ns["quantize_int8"])
        except (AssertionError, ValueError, OverflowError, FloatingPointError):
            failures += 1
    assert failures > 0, f"mutant '{name}' passed every pin"
