"""GPU parity: the HIP library, called through its C ABI, against the CPU
oracle on the same seeded inputs.  The bar is bit-exactness of both the
INT32 accumulators and the FP32 outputs (one scale multiply per output).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03026_amd import workloads as wl
from tests.golden.load import load_hand_example

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_03026_amd import _binding
    return _binding


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dmask(m):
    return dev(np.ascontiguousarray(m, dtype=np.uint64).view(np.int64))


def bits32(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def gpu_forward(sp, h, masks, B=None):
    B = masks.shape[0] if B is None else B
    out = torch.full((max(B, 1), h.N), float("nan"), dtype=torch.float32, device="cuda")
    sp.spike_proj_forward(h, dmask(masks), B, out)
    torch.cuda.synchronize()
    return out[:B].cpu().numpy()


def gpu_acc(sp, h, masks):
    B = masks.shape[0]
    acc = torch.full((B, h.N), -7, dtype=torch.int32, device="cuda")
    sp.spike_proj_forward_acc(h, dmask(masks), B, acc)
    torch.cuda.synchronize()
    return acc.cpu().numpy()


def assert_parity(sp, h, W, scale, masks, threads=8):
    ref_acc = oracle.spike_acc(W, masks)
    ref_out = oracle.spike_forward(W, scale, masks, threads=threads)
    got_acc = gpu_acc(sp, h, masks)
    got_out = gpu_forward(sp, h, masks)
    np.testing.assert_array_equal(got_acc, ref_acc)
    mism = bits32(got_out) != bits32(ref_out)
    assert not mism.any(), f"{int(mism.sum())} FP32 outputs differ, first at {np.argwhere(mism)[0]}"


def make(sp, W, scale):
    Wd, sd = dev(W), dev(scale)
    return sp.spike_proj_create(Wd, sd), Wd, sd


# Launch shapes exercised for every small case: (vector bytes per lane, mask
# words per K-slice); 0 means the automatic choice.
SHAPES = [(0, 0), (1, 1), (0, 1), (4, 3)]


def apply_shape(sp, h, vec, sw):
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_GATHER)
    if vec:
        try:
            sp.spike_proj_tune(h, sp.SPIKE_TUNE_VEC, vec)
        except sp.SpikeError:
            return False
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_SLICE_WORDS, sw)
    return True


def test_hand_worked_example(sp):
    g = load_hand_example()
    h, *_ = make(sp, g["W"], g["scale"])
    for vec, sw in SHAPES:
        if not apply_shape(sp, h, vec, sw):
            continue
        np.testing.assert_array_equal(gpu_acc(sp, h, g["masks"]), g["acc"])
        np.testing.assert_array_equal(bits32(gpu_forward(sp, h, g["masks"])), g["out_bits"])


@pytest.mark.parametrize("K", [1, 63, 64, 65, 200, 1000, 4097])
@pytest.mark.parametrize("N", [1, 7, 64, 100, 512, 1000, 1536])
def test_small_shapes(sp, K, N):
    p = wl.small_problem(K, N, 5, 0.3, seed=K + 7 * N)
    h, *_ = make(sp, p["W"], p["scale"])
    for vec, sw in SHAPES:
        if apply_shape(sp, h, vec, sw):
            assert_parity(sp, h, p["W"], p["scale"], p["masks"])


@pytest.mark.parametrize("vec", [16, 8, 4, 1])
def test_every_vector_width_on_the_decode_shape(sp, vec):
    d = wl.single_projection(n_masks=6)
    h, *_ = make(sp, d["W"], d["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_GATHER)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_VEC, vec)
    for sw in (0, 1, 5, 24):
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_SLICE_WORDS, sw)
        assert_parity(sp, h, d["W"], d["scale"], d["masks"])


PATHS = ["auto", "gather"]


def set_path(sp, h, path):
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_GATHER if path == "gather" else sp.SPIKE_PATH_AUTO)


@pytest.mark.parametrize("path", PATHS)
def test_single_projection_batch1(sp, path):
    """1536 -> 1536, Bernoulli(0.10): independent batch-1 calls, then one
    batch; on the automatic path (matrix cores) and on the gather."""
    d = wl.single_projection(n_masks=32)
    h, *_ = make(sp, d["W"], d["scale"])
    set_path(sp, h, path)
    ref = oracle.spike_forward(d["W"], d["scale"], d["masks"])
    for i in range(32):
        got = gpu_forward(sp, h, d["masks"][i:i + 1])
        np.testing.assert_array_equal(bits32(got), bits32(ref[i:i + 1]))
    assert_parity(sp, h, d["W"], d["scale"], d["masks"])


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("p", wl.DOWN_SWEEP_RATES)
def test_down_projection_sweep(sp, p, path):
    d = wl.down_sweep(p, n_masks=8)
    h, *_ = make(sp, d["W"], d["scale"])
    set_path(sp, h, path)
    ref = oracle.spike_forward(d["W"], d["scale"], d["masks"])
    for i in range(8):
        np.testing.assert_array_equal(bits32(gpu_forward(sp, h, d["masks"][i:i + 1])), bits32(ref[i:i + 1]))
    assert_parity(sp, h, d["W"], d["scale"], d["masks"])


@pytest.fixture(scope="module")
def stack(sp):
    """All 44 projections of the 22-block decode stack on the device."""
    hs, host = [], []
    for (l, j) in wl.stack_order():
        W, s = wl.stack_projection(l, j)
        h, Wd, sd = make(sp, W, s)
        hs.append(h)
        host.append((W, s))
    return hs, host


@pytest.mark.parametrize("path", PATHS)
def test_stack_driver_in_order(sp, stack, path):
    hs, host = stack
    for h in hs:
        set_path(sp, h, path)
    T = 3
    masks = wl.stack_token_masks(T)
    per_tok_out = sum(h.N for h in hs)
    for t in range(T):
        out = torch.full((per_tok_out,), float("nan"), device="cuda")
        sp.spike_stack_forward(hs, dmask(masks[t]), 1, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        moff = ooff = 0
        for h, (W, s) in zip(hs, host):
            wpr = wl.words_per_row(h.K)
            ref = oracle.spike_forward(W, s, masks[t:t + 1, moff:moff + wpr])[0]
            np.testing.assert_array_equal(bits32(got[ooff:ooff + h.N]), bits32(ref))
            moff += wpr
            ooff += h.N
    for h in hs:
        set_path(sp, h, "auto")


@pytest.mark.parametrize("n_sets", [1, 2])
def test_stream_small(sp, stack, n_sets):
    hs, host = stack
    if n_sets == 2:  # a second, address-distinct copy of every weight
        copies = [make(sp, W, s)[0] for (W, s) in host]
        hs_all, host_all = hs + copies, host + host
    else:
        hs_all, host_all = hs, host
    T = 5
    masks = wl.stack_token_masks(T)
    st = sp.spike_stream_create(hs_all, 44, n_sets, T)
    out = torch.full((T, 44 * 1536), float("nan"), device="cuda")
    sp.spike_stream_forward(st, dmask(masks), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    for t in range(T):
        moff = 0
        for j, (W, s) in enumerate(host_all[:44]):
            wpr = wl.words_per_row(W.shape[0])
            ref = oracle.spike_forward(W, s, masks[t:t + 1, moff:moff + wpr])[0]
            np.testing.assert_array_equal(bits32(got[t, j * 1536:(j + 1) * 1536]), bits32(ref))
            moff += wpr


def test_stream_full_workload(sp, stack):
    """The benchmark's configuration: 1000 tokens x 44 projections in one
    launch of the benchmark's stream kernel over 32 rotated weight copies;
    every one of the 44,000 (token, projection) outputs is checked against
    the oracle (one oracle call per projection over all 1000 rows)."""
    import bench
    hs, host = stack
    n_sets = bench.DEFAULT_SETS
    extra = []
    for _ in range(n_sets - 1):
        for h in hs:  # address-distinct device copies of the same weights
            extra.append(sp.spike_proj_create_reserved(h.W.clone(), h.scale.clone(), 1, gather_only=True))
    T = 1000
    masks = wl.stack_token_masks(T)
    st = sp.spike_stream_create(hs + extra, 44, n_sets, T)
    sp.spike_stream_tune(st, sp.SPIKE_TUNE_SHAPE, sp.SPIKE_SHAPE(*bench.HEADLINE_SHAPE))
    out = torch.full((T, 44 * 1536), float("nan"), device="cuda")
    sp.spike_stream_forward(st, dmask(masks), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    offs = np.cumsum([0] + [wl.words_per_row(W.shape[0]) for (W, _) in host])
    for j, (W, s) in enumerate(host):
        ref = oracle.spike_forward(W, s, masks[:, offs[j]:offs[j + 1]], threads=16)
        mism = bits32(got[:, j * 1536:(j + 1) * 1536]) != bits32(ref)
        assert not mism.any(), f"projection {j}: {int(mism.sum())} outputs differ, first at {np.argwhere(mism)[0]}"
    st.close()
    for c in extra:
        c.close()


def test_prefill_batch(sp):
    """512 tokens x 6144 -> 1536, Markov spikes at rate 0.10."""
    d = wl.prefill_projection()
    h, *_ = make(sp, d["W"], d["scale"])
    for path in (sp.SPIKE_PATH_GATHER, sp.SPIKE_PATH_AUTO):
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, path)
        assert_parity(sp, h, d["W"], d["scale"], d["masks"])


@pytest.fixture(scope="module")
def batched_stack(sp):
    hs, host = [], []
    for (l, j) in wl.stack_order():
        W, s = wl.batched_stack_projection(l, j)
        hs.append(make(sp, W, s)[0])
        host.append((W, s))
    bits = [wl.batched_stack_bits(l, j, B=64, n_steps=2) for (l, j) in wl.stack_order()]
    return hs, host, bits


@pytest.mark.parametrize("fused", [False, True])
def test_batched_decode_stack(sp, batched_stack, fused):
    """B = 64 rows through all 44 projections, structured spikes, two steps:
    in stream order (one launch per projection) and fused (one launch)."""
    hs, host, bits = batched_stack
    for step in range(2):
        masks = np.concatenate([wl.pack_bits(b[step]).reshape(-1) for b in bits])
        out = torch.full((sum(64 * h.N for h in hs),), float("nan"), device="cuda")
        (sp.spike_stack_forward_fused if fused else sp.spike_stack_forward)(hs, dmask(masks), 64, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        ooff = 0
        for (W, s), b in zip(host, bits):
            ref = oracle.spike_forward(W, s, wl.pack_bits(b[step]), threads=8)
            np.testing.assert_array_equal(bits32(got[ooff:ooff + ref.size]), bits32(ref.reshape(-1)))
            ooff += ref.size


@pytest.mark.parametrize("B", [5, 17, 64, 130])
def test_fused_stack_ragged(sp, B):
    """Fused launch over projections of different K (ragged K and B, junk
    padding bits past K) against the oracle, and against the in-order driver."""
    shapes = [(100, 96), (1536, 96), (70, 96), (4097, 96)]
    hs, host, ms = [], [], []
    for i, (K, N) in enumerate(shapes):
        p = wl.small_problem(K, N, B, 0.2, seed=100 + i)
        m = p["masks"].copy()
        if K % 64:
            m[:, -1] |= np.uint64(~((1 << (K % 64)) - 1) & 0xFFFFFFFFFFFFFFFF)  # junk past K
        hs.append(make(sp, p["W"], p["scale"])[0])
        host.append((p["W"], p["scale"]))
        ms.append(m)
    masks = np.concatenate([m.reshape(-1) for m in ms])
    n_out = sum(B * N for _, N in shapes)
    out_f = torch.full((n_out,), float("nan"), device="cuda")
    out_s = torch.full((n_out,), float("nan"), device="cuda")
    sp.spike_stack_forward_fused(hs, dmask(masks), B, out_f)
    sp.spike_stack_forward(hs, dmask(masks), B, out_s)
    torch.cuda.synchronize()
    got = out_f.cpu().numpy()
    assert np.array_equal(bits32(got), bits32(out_s.cpu().numpy()))
    ooff = 0
    for (W, s), m in zip(host, ms):
        ref = oracle.spike_forward(W, s, m, threads=8)
        np.testing.assert_array_equal(bits32(got[ooff:ooff + ref.size]), bits32(ref.reshape(-1)))
        ooff += ref.size


def test_fused_stack_refusals(sp):
    """The fused launch refuses what it cannot run, before any launch."""
    a = wl.small_problem(128, 64, 8, 0.2, seed=1)
    b = wl.small_problem(128, 32, 8, 0.2, seed=2)
    ha, hb = make(sp, a["W"], a["scale"])[0], make(sp, b["W"], b["scale"])[0]
    out = torch.empty(8 * 96, device="cuda")
    masks = dmask(np.concatenate([a["masks"].reshape(-1), b["masks"].reshape(-1)]))
    with pytest.raises(sp.SpikeError) as ei:
        sp.spike_stack_forward_fused([ha, hb], masks, 8, out)  # different N
    assert ei.value.code == sp.SPIKE_EUNSUPPORTED
    c = wl.small_problem(128, 64, 8, 0.2, seed=3)
    hc = sp.spike_proj_create_reserved(dev(c["W"]), dev(c["scale"]), 4, gather_only=True)  # no matrix-core copy
    with pytest.raises(sp.SpikeError) as ei:
        sp.spike_stack_forward_fused([ha, hc], masks, 4, out)
    assert ei.value.code == sp.SPIKE_EUNSUPPORTED


def test_batch_zero_is_a_noop(sp):
    p = wl.small_problem(100, 64, 1, 0.5)
    h, *_ = make(sp, p["W"], p["scale"])
    out = torch.full((1, 64), 3.0, device="cuda")
    sp.spike_proj_forward(h, dmask(p["masks"]), 0, out)
    torch.cuda.synchronize()
    assert (out == 3.0).all()


@pytest.mark.parametrize("K,N", [(1536, 1536), (6144, 1536), (77, 33)])
def test_degenerate_spike_patterns(sp, K, N):
    rng = np.random.default_rng(K)
    W = rng.integers(-128, 127, size=(K, N), dtype=np.int8, endpoint=True)
    scale = wl.uniform_scales(rng, N)
    bits = np.zeros((4, K), bool)
    bits[1] = True                      # all active
    bits[2, K - 1] = True               # only the last column
    bits[3, 0] = True                   # only the first column
    masks = wl.pack_bits(bits)
    if K % 64:                          # junk in the padding bits of every row
        masks[:, -1] |= np.uint64((~((1 << (K % 64)) - 1)) & 0xFFFFFFFFFFFFFFFF)
    h, *_ = make(sp, W, scale)
    for vec, sw in SHAPES:
        if apply_shape(sp, h, vec, sw):
            assert_parity(sp, h, W, scale, masks)
    out = gpu_forward(sp, h, masks[:1])
    assert not bits32(out).any()        # +0.0 for an empty spike set


def test_extreme_values(sp):
    """-128 weights, subnormal and tiny scales (no flush to zero)."""
    K, N = 1024, 256
    W = np.full((K, N), -128, np.int8)
    W[:, 1::2] = 127
    scale = np.full(N, 2.0 ** -140, np.float32)
    scale[::3] = 2.0 ** -149
    scale[1::5] = 1e-2
    masks = wl.pack_bits(np.ones((2, K), bool))
    h, *_ = make(sp, W, scale)
    assert_parity(sp, h, W, scale, masks)
    out = gpu_forward(sp, h, masks[:1])
    assert bits32(out).any()


@pytest.mark.parametrize("case", ["int32_min", "above_2_24"])
def test_maximum_K(sp, case):
    """K = 2^24 (the largest accepted): the INT32 sum reaches -2^31 exactly,
    and a sum of 2^24 + 1 must round to nearest even in the conversion."""
    K, N = 1 << 24, 1
    if case == "int32_min":
        W = np.full((K, N), -128, np.int8)
    else:
        W = np.ones((K, N), np.int8)
        W[0, 0] = 2
    scale = np.array([0.5], np.float32)
    masks = wl.pack_bits(np.ones((1, K), bool))
    h, *_ = make(sp, W, scale)
    ref = oracle.spike_acc(W, masks)
    assert ref[0, 0] == (-(1 << 31) if case == "int32_min" else (1 << 24) + 1)
    assert_parity(sp, h, W, scale, masks)


def test_repeat_runs_are_bit_identical(sp):
    d = wl.down_sweep(0.2, n_masks=4)
    h, *_ = make(sp, d["W"], d["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_GATHER)
    ref = bits32(oracle.spike_forward(d["W"], d["scale"], d["masks"]))
    for sw in (0, 1, 2, 7, 96):
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_SLICE_WORDS, sw)
        for _ in range(4):
            np.testing.assert_array_equal(bits32(gpu_forward(sp, h, d["masks"])), ref)


def test_workspace_resets_between_calls(sp):
    """Back-to-back split-K calls on one handle with changing B: a workspace
    or counter left dirty by one call would corrupt the next."""
    d = wl.down_sweep(0.1, n_masks=40)
    h, *_ = make(sp, d["W"], d["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_GATHER)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_SLICE_WORDS, 1)
    ref = oracle.spike_forward(d["W"], d["scale"], d["masks"])
    outs, lo = [], 0
    stream_out = []
    for B in (1, 7, 3, 16, 1, 12):
        out = torch.empty((B, 1536), device="cuda")
        sp.spike_proj_forward(h, dmask(d["masks"][lo:lo + B]), B, out)   # no sync between calls
        stream_out.append((lo, B, out))
        lo += B
    torch.cuda.synchronize()
    for lo, B, out in stream_out:
        np.testing.assert_array_equal(bits32(out.cpu().numpy()), bits32(ref[lo:lo + B]))


def test_row_major_weights_fail_parity(sp):
    """Passing the row-major [N, K] bytes where the column-major [K, N] layout
    is expected (K != N) must show up as a parity failure."""
    K, N = 96, 64
    p = wl.small_problem(K, N, 4, 0.4, seed=1)
    wrong = np.ascontiguousarray(p["W"].T).reshape(K, N)  # same bytes count, row-major order
    h, *_ = make(sp, wrong, p["scale"])
    got = gpu_forward(sp, h, p["masks"])
    ref = oracle.spike_forward(p["W"], p["scale"], p["masks"])
    assert (bits32(got) != bits32(ref)).any()


@pytest.mark.parametrize("path", PATHS)
def test_side_stream_and_graph_replay(sp, path):
    hs, host = [], []
    for K in (1536, 6144, 1536):
        p = wl.small_problem(K, 1536, 1, 0.1, seed=K)
        hs.append(make(sp, p["W"], p["scale"])[0])
        set_path(sp, hs[-1], path)
        host.append((p["W"], p["scale"]))
    words = sum(wl.words_per_row(h.K) for h in hs)
    static_mask = torch.zeros(words, dtype=torch.int64, device="cuda")
    static_out = torch.zeros(3 * 1536, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm up on a non-default stream
        sp.spike_stack_forward(hs, static_mask, 1, static_out)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sp.spike_stack_forward(hs, static_mask, 1, static_out)
    rng = np.random.default_rng(3)
    for replay in range(4):
        bits = [rng.random((1, h.K)) < 0.15 for h in hs]
        m = np.concatenate([wl.pack_bits(b).reshape(-1) for b in bits])
        static_mask.copy_(dmask(m))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = static_out.cpu().numpy()
        for j, ((W, s), b) in enumerate(zip(host, bits)):
            ref = oracle.spike_forward(W, s, wl.pack_bits(b))[0]
            np.testing.assert_array_equal(bits32(got[j * 1536:(j + 1) * 1536]), bits32(ref), err_msg=f"replay {replay}")
        # eager work between replays on the same handles
        eager = torch.zeros(3 * 1536, device="cuda")
        sp.spike_stack_forward(hs, static_mask, 1, eager)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(bits32(eager.cpu().numpy()), bits32(got))


@pytest.mark.parametrize("K", [1, 64, 65, 1536, 6144, 20000])
def test_compaction_kernel(sp, K):
    rng = np.random.default_rng(K)
    bits = rng.random((6, K)) < np.array([0.0, 1.0, 0.02, 0.1, 0.4, 0.9])[:, None]
    masks = wl.pack_bits(bits)
    if K % 64:
        masks[:, -1] |= np.uint64((~((1 << (K % 64)) - 1)) & 0xFFFFFFFFFFFFFFFF)
    idx = torch.full((6, K), -1, dtype=torch.int32, device="cuda")
    cnt = torch.full((6,), -1, dtype=torch.int32, device="cuda")
    sp.spike_compact(dmask(masks), 6, K, idx, cnt)
    torch.cuda.synchronize()
    idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
    for b in range(6):
        ref = oracle.active_indices(masks[b], K)
        assert cnt[b] == len(ref)
        np.testing.assert_array_equal(idx[b, :cnt[b]], ref)


def test_errors_on_gpu(sp):
    p = wl.small_problem(128, 64, 1, 0.5)
    h, *_ = make(sp, p["W"], p["scale"])
    out = torch.empty((600, 64), device="cuda")
    masks = torch.zeros((600, 2), dtype=torch.int64, device="cuda")
    with pytest.raises(sp.SpikeError) as e:
        sp.spike_proj_forward(h, masks, 513, out)
    assert e.value.code == sp.SPIKE_EINVAL
    sp.spike_proj_reserve(h, 600)
    sp.spike_proj_forward(h, masks, 600, out)
    torch.cuda.synchronize()
    assert not bits32(out.cpu().numpy()).any()
    for key, val in ((sp.SPIKE_TUNE_PATH, 9), (sp.SPIKE_TUNE_SLICE_WORDS, 257), (sp.SPIKE_TUNE_VEC, 3), (99, 0)):
        with pytest.raises(sp.SpikeError):
            sp.spike_proj_tune(h, key, val)
    q = wl.small_problem(128, 32, 1, 0.5)
    h2, *_ = make(sp, q["W"], q["scale"])
    with pytest.raises(sp.SpikeError) as e:
        sp.spike_stream_create([h, h2], 2, 1, 4)
    assert e.value.code == sp.SPIKE_EUNSUPPORTED


def decode_shape(code):
    return dict(V=code & 31, LG=(code >> 5) & 1023, U=(code >> 15) & 31, BLOCK=((code >> 20) & 31) * 64,
                NT=bool(code >> 25 & 1), I16=bool(code >> 26 & 1))


@pytest.mark.parametrize("weights", ["min", "max", "random"])
@pytest.mark.parametrize("p,slice_words", [(1.0, 256), (1.0, 100), (0.6, 256)])
def test_int16_partials_fold_exactly(sp, weights, p, slice_words):
    """The 16-bit partial-sum shape over long dense rows: every lane adds
    thousands of columns, so the biased 16-bit halves are folded into INT32
    many times, at the extremes of the weight range too."""
    K, N, B = 16384, 512, 2
    code = sp.SPIKE_SHAPE(16, 32, 4, 256, NT=True, I16=True)
    assert code in sp.spike_proj_shapes()
    q = wl.small_problem(K, N, B, p, seed=11)
    W = {"min": np.full((K, N), -128, np.int8), "max": np.full((K, N), 127, np.int8), "random": q["W"]}[weights]
    h, *_ = make(sp, W, q["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_GATHER)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_SHAPE, code)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_SLICE_WORDS, slice_words)
    assert_parity(sp, h, W, q["scale"], q["masks"], threads=16)


@pytest.mark.parametrize("K,N", [(1536, 1536), (6144, 1536), (333, 1000), (70, 96)])
def test_every_instantiated_shape(sp, K, N):
    """Every launch shape the library instantiates, with and without K-slices
    and with several tiles per workgroup, gives the oracle's bits."""
    p = wl.small_problem(K, N, 3, 0.2, seed=K ^ N)
    h, *_ = make(sp, p["W"], p["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_GATHER)
    wpr = wl.words_per_row(K)
    ran = 0
    for code in sp.spike_proj_shapes():
        try:
            sp.spike_proj_tune(h, sp.SPIKE_TUNE_SHAPE, code)
        except sp.SpikeError:
            assert N % decode_shape(code)["V"] != 0  # only a misfit vector width may be refused
            continue
        for sw, tpu in ((wpr, 1), (max(1, wpr // 3), 1), (1, 3)):
            sp.spike_proj_tune(h, sp.SPIKE_TUNE_SLICE_WORDS, min(sw, 256))
            sp.spike_proj_tune(h, sp.SPIKE_TUNE_TILES_PER_UNIT, tpu)
            assert_parity(sp, h, p["W"], p["scale"], p["masks"])
        ran += 1
    assert ran == sum(N % decode_shape(c)["V"] == 0 for c in sp.spike_proj_shapes())


def test_stream_every_shape_and_xcd_spread(sp, stack):
    hs, host = stack
    T = 3
    masks = wl.stack_token_masks(T)
    st = sp.spike_stream_create(hs, 44, 1, T)
    ref = torch.full((T, 44 * 1536), float("nan"), device="cuda")
    sp.spike_stream_forward(st, dmask(masks), ref)
    torch.cuda.synchronize()
    got_ref = ref.cpu().numpy()
    moff = 0
    for j, (W, s) in enumerate(host):  # the default shape against the oracle, every token
        wpr = wl.words_per_row(W.shape[0])
        np.testing.assert_array_equal(bits32(got_ref[:, j * 1536:(j + 1) * 1536]),
                                      bits32(oracle.spike_forward(W, s, masks[:, moff:moff + wpr])))
        moff += wpr
    for code in sp.spike_proj_shapes():
        for tpu in (1, 2):
            for spread in (1, 8):
                sp.spike_stream_tune(st, sp.SPIKE_TUNE_SHAPE, code)
                sp.spike_stream_tune(st, sp.SPIKE_TUNE_TILES_PER_UNIT, tpu)
                sp.spike_stream_tune(st, sp.SPIKE_TUNE_XCD_SPREAD, spread)
                out = torch.full_like(ref, float("nan"))
                sp.spike_stream_forward(st, dmask(masks), out)
                torch.cuda.synchronize()
                assert torch.equal(out.view(torch.int32), ref.view(torch.int32)), (hex(code), tpu, spread)


@pytest.mark.parametrize("B", [1, 17, 64, 65, 130])
@pytest.mark.parametrize("K,N", [(100, 64), (1536, 1536), (4097, 192), (6144, 1024)])
def test_matrix_core_path(sp, B, K, N):
    """The dense i8 matrix-core contraction over the 0/1 spike matrix gives the
    oracle's bits with its automatic plan and with 4, 8 and 16 waves, for
    ragged B and K."""
    p = wl.small_problem(K, N, B, 0.15, seed=B * 7 + K)
    h, *_ = make(sp, p["W"], p["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_MFMA)
    assert_parity(sp, h, p["W"], p["scale"], p["masks"])
    wpr = wl.words_per_row(K)
    for waves in (4, 8, 16):
        if waves > wpr:
            continue
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_MFMA_WAVES, waves)
        try:
            assert_parity(sp, h, p["W"], p["scale"], p["masks"])
        except sp.SpikeError as e:  # that wave count has no instantiated plan for this shape
            assert e.code == sp.SPIKE_EUNSUPPORTED


def plan_shape(plan, seed):
    """A ragged shape that the given matrix-core plan can run: K past a
    multiple of 64, B past a row-tile multiple, N over a number of tiles that
    is not a multiple of 8 (plain tile order) for odd seeds."""
    rt, cs, kw, d = plan["rt"], plan["cs"], plan["kw"], plan["d"]
    if plan["preload"]:
        wpr = max(kw, kw * d - 1)
    else:
        wpr = kw * d * 2 + 3
    stage_words = (64 * 1024 - rt * cs * 1024) // (128 * rt)
    wpr = min(wpr, stage_words - 1)
    K = 64 * (wpr - 1) + 37
    coltiles = 8 if seed % 2 == 0 else 5
    N = 16 * cs * coltiles
    B = 16 * rt + 16 * rt // 2 + 3
    return K, N, B


def test_every_matrix_core_plan(sp):
    """Every instantiated matrix-core plan (tile height and width, waves,
    weight depth, preloaded or ring) against the oracle, on a shape it runs."""
    plans = [p for p in sp.spike_mfma_plans() if not p["direct"]]  # direct plans: next test
    assert len(plans) >= 30
    for i, plan in enumerate(plans):
        K, N, B = plan_shape(plan, i)
        wpr = wl.words_per_row(K)
        steps = -(-wpr // plan["kw"])
        assert wpr >= plan["kw"] and (steps <= plan["d"]) == plan["preload"], (plan, K)
        p = wl.small_problem(K, N, B, 0.2, seed=i)
        masks = p["masks"].copy()
        masks[:, -1] |= np.uint64((~((1 << (K % 64)) - 1)) & 0xFFFFFFFFFFFFFFFF)  # junk past K
        h, *_ = make(sp, p["W"], p["scale"])
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_MFMA)
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_MFMA_ROW_TILE, plan["rt"])
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_MFMA_COL_SETS, plan["cs"])
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_MFMA_WAVES, plan["kw"])
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_MFMA_DEPTH, plan["d"])
        print(f"plan {plan} K={K} N={N} B={B}", flush=True)
        assert_parity(sp, h, p["W"], p["scale"], masks)
        h.close()


def test_direct_spike_loads_for_the_smallest_batches(sp):
    """Batches of at most 4 rows load their spike words with each k-step
    instead of staging them: every direct plan (K from one word to past 2048,
    every preload depth and the ring past 6144) against the oracle, with junk bits
    past K, for 1 to 4 rows and channel counts that are and are not a
    multiple of 8 channel sets."""
    direct = {tuple(p.values()) for p in sp.spike_mfma_plans() if p["direct"]}
    assert len(direct) >= 5
    seen = set()
    for K in (40, 150, 300, 512, 1000, 1536, 1900, 2111, 6144, 6400):
        for N in (48, 1536):
            for B in (1, 2, 3, 4):
                path, plan = sp.spike_proj_plan_query(K, N, B)
                assert path == sp.SPIKE_PATH_MFMA and plan["direct"], (K, N, B, plan)
                seen.add(tuple(plan.values()))
                p = wl.small_problem(K, N, B, 0.2, seed=K + N + B)
                masks = p["masks"].copy()
                if K % 64:
                    masks[:, -1] |= np.uint64((~((1 << (K % 64)) - 1)) & 0xFFFFFFFFFFFFFFFF)
                h, *_ = make(sp, p["W"], p["scale"])
                assert_parity(sp, h, p["W"], p["scale"], masks)
                h.close()
    assert seen == direct, (seen, direct)
    # from 5 rows on, the staged plans
    assert not sp.spike_proj_plan_query(1536, 1536, 5)[1]["direct"]


def test_matrix_core_extremes(sp):
    K, N = 2048, 128
    W = np.full((K, N), -128, np.int8)
    W[:, ::3] = 127
    scale = np.full(N, 2.0 ** -140, np.float32)
    scale[1::4] = 1e-2
    bits = np.ones((70, K), bool)
    bits[3] = False
    masks = wl.pack_bits(bits)
    h, *_ = make(sp, W, scale)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_MFMA)
    assert_parity(sp, h, W, scale, masks)
    assert_parity(sp, h, W, scale, masks[:9])


def test_matrix_core_rejects_unaligned_N(sp):
    p = wl.small_problem(128, 100, 4, 0.3)
    h, *_ = make(sp, p["W"], p["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_MFMA)
    out = torch.empty((4, 100), device="cuda")
    with pytest.raises(sp.SpikeError) as e:
        sp.spike_proj_forward(h, dmask(p["masks"]), 4, out)
    assert e.value.code == sp.SPIKE_EUNSUPPORTED
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_AUTO)  # AUTO falls back to the gather
    assert_parity(sp, h, p["W"], p["scale"], p["masks"])


def test_auto_falls_back_when_the_plan_cannot_run(sp):
    """A tuned matrix-core plan that is not instantiated is refused when the
    matrix cores are forced, and AUTO serves the same call on the gather."""
    p = wl.small_problem(1536, 1536, 40, 0.1, seed=11)
    h, *_ = make(sp, p["W"], p["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_MFMA_ROW_TILE, 8)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_MFMA_COL_SETS, 6)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_MFMA)
    out = torch.empty((40, 1536), device="cuda")
    with pytest.raises(sp.SpikeError) as e:
        sp.spike_proj_forward(h, dmask(p["masks"]), 40, out)
    assert e.value.code == sp.SPIKE_EUNSUPPORTED and "instantiated" in str(e.value)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_AUTO)
    assert_parity(sp, h, p["W"], p["scale"], p["masks"])


def test_reserve_drops_and_remakes_the_matrix_core_copy(sp):
    """With the matrix-core minimum raised to 5 rows, reserve() below it
    frees the packed copy (the matrix cores then refuse, AUTO uses the
    gather); a larger reserve makes it again from W."""
    p = wl.small_problem(1000, 256, 20, 0.2, seed=5)
    h, *_ = make(sp, p["W"], p["scale"])
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_MFMA_MIN_B, 5)
    sp.spike_proj_reserve(h, 1)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_MFMA)
    out = torch.empty((1, 256), device="cuda")
    with pytest.raises(sp.SpikeError) as e:
        sp.spike_proj_forward(h, dmask(p["masks"][:1]), 1, out)
    assert e.value.code == sp.SPIKE_EUNSUPPORTED
    sp.spike_proj_reserve(h, 20)
    assert_parity(sp, h, p["W"], p["scale"], p["masks"])


def test_auto_path_at_a_million_channels(sp):
    """K = 1600, N = 2^20, B = 10: AUTO runs this on the matrix cores (plan
    query and result); 4096 sampled channels are checked against the oracle
    on the same columns of W."""
    K, N, B = 1600, 1 << 20, 10
    path, plan = sp.spike_proj_plan_query(K, N, B)
    assert path == sp.SPIKE_PATH_MFMA and plan is not None
    rng = np.random.default_rng(77)
    Wd = torch.randint(-127, 128, (K, N), dtype=torch.int8, device="cuda")
    sd = torch.rand(N, device="cuda") * 9e-3 + 1e-3
    bits = rng.random((B, K)) < 0.1
    masks = wl.pack_bits(bits)
    h = sp.spike_proj_create(Wd, sd)
    out = torch.empty((B, N), device="cuda")
    sp.spike_proj_forward(h, dmask(masks), B, out)
    torch.cuda.synchronize()
    sel = np.sort(rng.choice(N, 4096, replace=False))
    sel_t = torch.from_numpy(sel).cuda()
    Wsel = Wd[:, sel_t].cpu().numpy()
    ssel = sd[sel_t].cpu().numpy()
    ref = oracle.spike_forward(Wsel, ssel, masks, threads=8)
    got = out[:, sel_t].cpu().numpy()
    assert np.array_equal(bits32(got), bits32(ref))
    h.close()
    del Wd


@pytest.mark.parametrize("K", [100, 4097])
def test_matrix_core_padding_junk_and_unaligned_weights(sp, K):
    """Spike bits past K are ignored on the matrix-core path (they meet the
    zero padding of its packed weight copy), and W needs no alignment there:
    the copy is made once, at create, from a W that starts at an odd byte."""
    N, B = 192, 70
    p = wl.small_problem(K, N, B, 0.2, seed=K)
    masks = p["masks"].copy()
    masks[:, -1] |= np.uint64((~((1 << (K % 64)) - 1)) & 0xFFFFFFFFFFFFFFFF)
    buf = torch.zeros(K * N + 1, dtype=torch.int8, device="cuda")
    buf[1:].copy_(torch.from_numpy(p["W"].reshape(-1)))
    Wd, sd = buf[1:].view(K, N), dev(p["scale"])
    h = sp.spike_proj_create(Wd, sd)
    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, sp.SPIKE_PATH_MFMA)
    assert_parity(sp, h, p["W"], p["scale"], masks)  # tall tiles (B > 64)
    assert_parity(sp, h, p["W"], p["scale"], masks[:64])  # narrow tiles
    assert_parity(sp, h, p["W"], p["scale"], masks[:5])
    # the packed copy is taken at create: later writes to W are not seen by
    # the matrix cores (W is borrowed read-only for the handle's lifetime)
    Wd.zero_()
    torch.cuda.synchronize()
    assert_parity(sp, h, p["W"], p["scale"], masks)


def test_both_paths_on_prefill_spikes_with_padding_junk(sp):
    """Markov prefill spikes at a K that is not a multiple of 64, with every
    padding bit of the last word set: the gather and the matrix cores each
    match the oracle."""
    K, N, B = 6144 - 64 * 3 + 37, 1536, 200
    bits = wl.prefill_bits(B, K)
    masks = wl.pack_bits(bits)
    masks[:, -1] |= np.uint64((~((1 << (K % 64)) - 1)) & 0xFFFFFFFFFFFFFFFF)
    rng = np.random.default_rng([42, 9, 200])
    W = wl.uniform_weights(rng, K, N)
    scale = wl.uniform_scales(rng, N)
    h, *_ = make(sp, W, scale)
    for path in (sp.SPIKE_PATH_GATHER, sp.SPIKE_PATH_MFMA):
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, path)
        assert_parity(sp, h, W, scale, masks)
