"""Pins for the output-head candidate verification in the CPU oracle (no GPU).

Paper Sec. 5: INT8-activation head over all rows, top-two gap gate, FP32
recompute of the top K rows.  Checked against facts that do not come from the
oracle: a hand-worked example (tests/golden) where verification changes the
token, the activation quantizer's reconstruction bound, the approximate
logits against the exact product within the quantization error, the
candidate set checked by pairwise comparison (not by re-sorting), the gate's
limits (threshold 0 never verifies, +inf always does), integer-grid inputs
where INT8 activations are exact, and planted mistakes in a copy of the
oracle source.
"""
import numpy as np
import pytest

from oracle import head_oracle
from oracle.head_oracle import head_verify, quantize_activations
from tests.golden.load import load_head_example


def problem(V, K, seed):
    rng = np.random.default_rng([42, 15, V, K, seed])
    Q = np.clip(np.rint(rng.normal(0, 30, size=(V, K))), -127, 127).astype(np.int8)
    s = rng.uniform(1e-3, 1e-2, V).astype(np.float32)
    x = rng.standard_normal(K).astype(np.float32)
    return Q, s, x


def check_hand_example(mod):
    g = load_head_example()
    xq, sx = mod.quantize_activations(g["x"])
    assert sx == np.float32(1.0)
    np.testing.assert_array_equal(xq, g["xq"])
    np.testing.assert_array_equal(mod.approx_logits(g["Q"], g["scale"], g["x"]), g["logits"].astype(np.float32))
    np.testing.assert_array_equal(mod.top_candidates(mod.approx_logits(g["Q"], g["scale"], g["x"]), 5), g["order"])
    for k, thr, verified, token in g["case"]:
        r = mod.head_verify(g["Q"], g["scale"], g["x"], k, thr)
        assert r["gap"] == np.float32(g["gap"][0])
        assert (r["verified"], r["token"]) == (verified, token), (k, thr, r["verified"], r["token"])
        if verified:
            np.testing.assert_array_equal(r["recomputed"], g["recomputed"][r["cand"]])


def check_candidates_by_comparison(mod):
    """Every candidate beats every other row (larger logit, or equal and a
    lower row), and candidates are in that order; many exact ties."""
    rng = np.random.default_rng(3)
    logits = rng.integers(-20, 20, size=500).astype(np.float32) * np.float32(0.25)
    for k in (1, 2, 16, 64, 500):
        c = mod.top_candidates(logits, k)
        assert len(c) == k and len(set(c.tolist())) == k

        def better(a, b):
            return logits[a] > logits[b] or (logits[a] == logits[b] and a < b)
        rest = np.setdiff1d(np.arange(500), c)
        for i in range(k - 1):
            assert better(c[i], c[i + 1])
        if len(rest):
            worst = c[-1]
            assert all(better(worst, r) for r in rest)


def check_approx_error_bound(mod):
    """|approx - exact| <= s_m s_x / 2 sum_k |Q| (activation rounding) plus a
    few binary32 roundings of the result."""
    Q, s, x = problem(300, 512, 1)
    lo = mod.approx_logits(Q, s, x).astype(np.float64)
    exact = s.astype(np.float64) * (Q.astype(np.float64) @ x.astype(np.float64))
    _, sx = mod.quantize_activations(x)
    bound = s.astype(np.float64) * float(sx) / 2 * np.abs(Q.astype(np.float64)).sum(axis=1)
    assert (np.abs(lo - exact) <= bound * (1 + 1e-6) + 4 * 2.0 ** -24 * np.abs(lo)).all()


def check_gate_limits(mod):
    Q, s, x = problem(200, 256, 2)
    never = mod.head_verify(Q, s, x, 16, 0.0)
    always = mod.head_verify(Q, s, x, 16, np.inf)
    assert not never["verified"] and never["token"] == never["cand"][0]
    assert always["verified"]
    exact = s.astype(np.float64) * (Q.astype(np.float64) @ x.astype(np.float64))
    c = always["cand"]
    assert always["token"] == c[int(np.argmax(exact[c]))]
    assert never["gap"] >= 0


def check_integer_grid_is_exact(mod):
    """x on the INT8 grid with max |x| = 127 gives s_x = 1 and xq = x, so the
    approximate logits equal s_m * (Q x) rounded once (Q x exact in binary32)."""
    Q, s, _ = problem(100, 64, 4)
    rng = np.random.default_rng(5)
    x = rng.integers(-127, 128, size=64).astype(np.float32)
    x[7] = 127
    acc = Q.astype(np.int64) @ x.astype(np.int64)
    want = (acc.astype(np.float32) * s).astype(np.float32)
    np.testing.assert_array_equal(mod.approx_logits(Q, s, x), want)


def check_activation_quantizer(mod):
    x = np.random.default_rng(6).standard_normal(1000).astype(np.float32)
    xq, sx = mod.quantize_activations(x)
    assert np.abs(xq).max() == 127
    assert (np.abs(xq.astype(np.float64) * float(sx) - x) <= float(sx) * (0.5 + 2.0 ** -20)).all()
    zq, zs = mod.quantize_activations(np.zeros(9, dtype=np.float32))
    assert (zq == 0).all() and abs(float(zs) * 127 - 1e-8) < 1e-14


CHECKS = [check_hand_example, check_candidates_by_comparison, check_approx_error_bound, check_gate_limits,
          check_integer_grid_is_exact, check_activation_quantizer]


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_oracle_meets(check):
    check(head_oracle)


def test_single_row_and_argument_checks():
    Q, s, x = problem(1, 32, 7)
    r = head_verify(Q, s, x, 1, 0.5)
    assert r["gap"] == np.inf and r["token"] == 0 and not r["verified"]
    with pytest.raises(ValueError):
        head_verify(Q, s, x, 2, 0.5)
    with pytest.raises(ValueError):
        quantize_activations(np.zeros(3, dtype=np.float64))


MUTANTS = {
    "ties to the higher row": ("key=lambda m: (-float(logits[m]), m)", "key=lambda m: (-float(logits[m]), -m)"),
    "gap the wrong way": ("logits[top2[0]] - logits[top2[1]]", "logits[top2[1]] - logits[top2[0]]"),
    "gate at or below": ("gap < np.float32(threshold)", "gap <= np.float32(threshold)"),
    "activation truncation": ("np.rint(x / sx)", "np.trunc(x / sx)"),
    "weight scale only": ("(scale * sx).astype(np.float32)", "scale.astype(np.float32)"),
    "recompute token ignores verification": ("token = int(cand[best])", "token = int(cand[0])"),
    "recompute with INT8 activations": ("xd = np.asarray(x, dtype=np.float64)",
                                        "xd = quantize_activations(x)[0].astype(np.float64) * float(quantize_activations(x)[1])"),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistakes_are_caught(name):
    import types
    src = open(head_oracle.__file__).read()
    old, new = MUTANTS[name]
    assert old in src
    mod = types.ModuleType("mutant_head", None)
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    failures = 0
    for check in CHECKS:
        try:
            check(mod)
        except (AssertionError, ValueError):
            failures += 1
    assert failures > 0, f"mutant '{name}' passed every pin"
