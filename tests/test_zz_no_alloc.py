"""spike_proj_forward_noalloc: the handle-free forward on the library's
static scratch array, checked bit for bit against spike_proj_forward on a
handle over the same weights and against the CPU oracle, on two calls in a
row (the second smaller), with and without a K-split through the scratch."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03026_amd import workloads as wl

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


def handle_forward(sp, W, s, masks):
    h = sp.spike_proj_create(W, s)
    B = masks.shape[0]
    out = torch.full((B, h.N), float("nan"), device="cuda")
    sp.spike_proj_forward(h, dmask(masks), B, out)
    torch.cuda.synchronize()
    h.close()
    return out.cpu().numpy()


# (K, N, B first, B second): K = 6144 at B <= 4 and K = 40000 split K across
# workgroups (partial sums and counters in the scratch); the others do not.
CASES = [(6144, 1536, 4, 1), (1536, 1536, 3, 2), (40000, 192, 8, 3), (4097, 100, 3, 1), (1536, 1536, 16, 2),
         (64, 64, 5, 1)]


@pytest.mark.parametrize("K,N,B1,B2", CASES)
def test_two_calls_in_a_row_match_the_handle_path(sp, K, N, B1, B2):
    p1 = wl.small_problem(K=K, N=N, B=B1, p=0.1, seed=11)
    rng = np.random.default_rng([wl.SEED, wl.W_TESTS, K, N, B2, 12])
    m2 = wl.pack_bits(rng.random((B2, K)) < 0.3)
    W, s = dev(p1["W"]), dev(p1["scale"])
    o1 = torch.full((B1, N), float("nan"), device="cuda")
    o2 = torch.full((B2, N), float("nan"), device="cuda")
    d1, d2 = dmask(p1["masks"]), dmask(m2)
    sp.spike_proj_forward_noalloc(W, s, d1, B1, o1)
    sp.spike_proj_forward_noalloc(W, s, d2, B2, o2)  # same stream, no host sync in between
    torch.cuda.synchronize()
    for out, masks in ((o1, p1["masks"]), (o2, m2)):
        got = out.cpu().numpy()
        ref_handle = handle_forward(sp, W, s, masks)
        ref_oracle = oracle.spike_forward(p1["W"], p1["scale"], masks)
        assert np.array_equal(bits32(got), bits32(ref_handle))
        assert np.array_equal(bits32(got), bits32(ref_oracle))


def test_scratch_limit(sp):
    """B * (N + ceil(N/32)) words may fill the scratch exactly up to its size;
    one more row is refused before any launch."""
    K, N = 64, 1536
    cap = sp.SPIKE_STATIC_SCRATCH_WORDS
    B_max = cap // (N + (N + 31) // 32)
    p = wl.small_problem(K=K, N=N, B=B_max, p=0.2, seed=3)
    W, s = dev(p["W"]), dev(p["scale"])
    out = torch.full((B_max, N), float("nan"), device="cuda")
    sp.spike_proj_forward_noalloc(W, s, dmask(p["masks"]), B_max, out)
    torch.cuda.synchronize()
    assert np.array_equal(bits32(out.cpu().numpy()), bits32(oracle.spike_forward(p["W"], p["scale"], p["masks"])))
    big = torch.zeros((B_max + 1, wl.words_per_row(K)), dtype=torch.int64, device="cuda")
    out2 = torch.empty((B_max + 1, N), device="cuda")
    with pytest.raises(sp.SpikeError) as ei:
        sp.spike_proj_forward_noalloc(W, s, big, B_max + 1, out2)
    assert ei.value.code == sp.SPIKE_EINVAL and "scratch" in str(ei.value)


def test_graph_replays_with_eager_calls_between(sp):
    """A captured call replays correctly, with eager calls of other shapes
    using the same scratch in between."""
    K, N = 6144, 1536
    p = wl.small_problem(K=K, N=N, B=2, p=0.15, seed=5)
    q = wl.small_problem(K=K, N=N, B=3, p=0.05, seed=6)
    W, s = dev(p["W"]), dev(p["scale"])
    Wq, sq = dev(q["W"]), dev(q["scale"])
    dm, dq = dmask(p["masks"]), dmask(q["masks"])
    out = torch.zeros((2, N), device="cuda")
    outq = torch.zeros((3, N), device="cuda")
    ref = oracle.spike_forward(p["W"], p["scale"], p["masks"])
    refq = oracle.spike_forward(q["W"], q["scale"], q["masks"])
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        sp.spike_proj_forward_noalloc(W, s, dm, 2, out)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            sp.spike_proj_forward_noalloc(W, s, dm, 2, out)
    torch.cuda.synchronize()
    for _ in range(4):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits32(out.cpu().numpy()), bits32(ref))
        outq.fill_(float("nan"))
        sp.spike_proj_forward_noalloc(Wq, sq, dq, 3, outq)
        torch.cuda.synchronize()
        assert np.array_equal(bits32(outq.cpu().numpy()), bits32(refq))
