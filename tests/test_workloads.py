"""Seeded input generators: determinism, packing layout, and that each
workload's statistics match its recipe (no GPU needed)."""
import numpy as np
import pytest

from paper_2606_03026_amd import workloads as wl


@pytest.mark.parametrize("K", [1, 5, 63, 64, 65, 1536, 6144])
def test_pack_layout_matches_packbits_little(K):
    bits = np.random.default_rng(K).random((3, K)) < 0.5
    m = wl.pack_bits(bits)
    assert m.dtype == np.uint64 and m.shape == (3, wl.words_per_row(K))
    by = m.view(np.uint8)
    ref = np.packbits(bits, axis=1, bitorder="little")
    np.testing.assert_array_equal(by[:, : ref.shape[1]], ref)
    assert not by[:, ref.shape[1]:].any()
    np.testing.assert_array_equal(wl.unpack_bits(m, K), bits)
    # bit k is bit k % 64 of word k // 64
    for b in range(3):
        for k in map(int, np.flatnonzero(bits[b])[:20]):
            assert (int(m[b, k // 64]) >> (k % 64)) & 1


def test_generators_are_deterministic():
    a = wl.single_projection(n_masks=4)
    b = wl.single_projection(n_masks=4)
    for key in ("W", "scale", "masks"):
        np.testing.assert_array_equal(a[key], b[key])
    # a shorter run draws a prefix of a longer one
    np.testing.assert_array_equal(wl.stack_masks(3, 1, 5), wl.stack_masks(3, 1, 9)[:5])


def test_single_projection_recipe():
    d = wl.single_projection(n_masks=400)
    assert d["W"].shape == (1536, 1536) and d["W"].dtype == np.int8
    assert d["W"].min() >= -127 and d["W"].max() <= 127
    assert 1e-3 <= d["scale"].min() and d["scale"].max() <= 1e-2
    rate = wl.unpack_bits(d["masks"], 1536).mean()
    assert abs(rate - 0.10) < 0.005


@pytest.mark.parametrize("p", wl.DOWN_SWEEP_RATES)
def test_down_sweep_rates(p):
    d = wl.down_sweep(p, n_masks=64)
    assert d["W"].shape == (6144, 1536)
    rate = wl.unpack_bits(d["masks"], 6144).mean()
    assert abs(rate - p) < 0.01 + 0.05 * p


def test_stack_layout_and_rates():
    rates = wl.stack_layer_rates()
    assert rates.shape == (22,) and rates.min() >= 0.05 and rates.max() <= 0.20
    order = wl.stack_order()
    assert len(order) == 44 and order[:2] == [(0, 0), (0, 1)]
    m = wl.stack_token_masks(3, n_layers=2)
    assert m.shape == (3, 24 + 96 + 24 + 96)
    np.testing.assert_array_equal(m[:, 24:120], wl.stack_masks(0, 1, 3))
    W, s = wl.stack_projection(5, 1)
    assert W.shape == (6144, 1536) and s.shape == (1536,)


def test_prefill_markov_statistics():
    x = wl.prefill_bits()
    assert x.shape == (512, 6144)
    assert abs(x.mean() - 0.10) < 0.01
    prev, nxt = x[:-1], x[1:]
    stay = (prev & nxt).sum() / prev.sum()
    assert abs(stay - 0.5) < 0.02
    flip = (prev != nxt).mean()
    assert abs(flip - 0.10) < 0.01


def test_batched_stack_statistics():
    bits = wl.batched_stack_bits(0, 1, B=64, n_steps=4)
    assert bits.shape == (4, 64, 6144)
    col_rate = bits.mean(axis=(0, 1))
    hot = col_rate > 0.6
    assert hot.sum() == round(0.05 * 6144)
    assert abs(bits[:, :, ~hot].mean() - 0.10) < 0.03
    W, _ = wl.batched_stack_projection(0, 1)
    assert W.min() >= -127 and W.max() <= 127 and abs(W.std() - 30) < 1.5
