"""GPU parity of the dense continuous-input INT8 projection (dense_proj.h)
against the CPU oracle's float64 definition.

FP32 accumulation is not associative, so outside integer inputs the bar is
the forward error bound of the kernel's fixed summation order: with
u = 2^-24, gamma(n) = n u / (1 - n u) and h = ceil(K/16) + 20 (a per-lane
FMA chain of at most ceil(K/16) + 15 products, a lane tree of at most 5
levels, one slack level),

    |y - exact| <= u |exact| + (1 + u) s_m gamma(h) sum_k |Q[m,k] x[b,k]|.

The oracle computes `exact` in float64 (its own rounding is below 2^-40
relative at these sizes and is covered by the slack level).  With integer
inputs every partial sum is an exact FP32 integer, so y must equal the
correctly rounded product bit for bit.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_03026_amd import workloads as wl

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(scope="module")
def sp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_03026_amd import _binding
    return _binding


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def bits32(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def q_at(Q, offset):
    """Device copy of Q whose first byte sits `offset` bytes past a 256-byte
    aligned allocation (selects the 16-, 4- or 1-byte load path)."""
    M, K = Q.shape
    buf = torch.zeros(M * K + 256, dtype=torch.int8, device="cuda")
    view = buf[offset:offset + M * K].view(M, K)
    view.copy_(torch.from_numpy(np.ascontiguousarray(Q)))
    return view


def run(sp, Q, scale, x, B=None, q_offset=0):
    B = x.shape[0] if B is None else B
    M = Q.shape[0]
    y = torch.full((max(B, 1), M), float("nan"), dtype=torch.float32, device="cuda")
    sp.dense_proj_forward(q_at(Q, q_offset), dev(scale), dev(x), B, y)
    torch.cuda.synchronize()
    return y[:B].cpu().numpy()


def bound(Q, scale, x, exact):
    K = Q.shape[1]
    h = math.ceil(K / 16) + 20
    gamma = h * U / (1 - h * U)
    absdot = np.abs(x.astype(np.float64)) @ np.abs(Q.astype(np.float64)).T
    return U * np.abs(exact) + (1 + U) * scale.astype(np.float64)[None, :] * gamma * absdot


def assert_within_bound(got, Q, scale, x):
    exact = oracle.dense_forward(Q, scale, x)
    assert got.shape == exact.shape
    assert np.isfinite(got).all(), "non-finite outputs (rows left unwritten?)"
    err = np.abs(got.astype(np.float64) - exact)
    lim = bound(Q, scale, x, exact)
    bad = err > lim
    assert not bad.any(), (f"{int(bad.sum())} outputs outside the FP32 bound; first at {np.argwhere(bad)[0]}: "
                           f"err {err[bad][0]:.3e} > {lim[bad][0]:.3e}")
    return float((err / np.maximum(lim, 1e-300)).max())


# (M, K): ragged row counts (not multiples of 16 rows, of the rows per
# workgroup, or of a whole ring round), one-row and one-column edges, and the
# largest K the staged activations allow.
SHAPES = [(1, 1), (5, 17), (16, 16), (33, 100), (100, 64), (257, 1536), (1000, 1540), (4097, 96),
          (2053, 272), (64, 16128), (3, 16127)]


@pytest.mark.parametrize("M,K", SHAPES)
@pytest.mark.parametrize("B", [1, 3, 8, 13])
def test_dense_matches_oracle(sp, M, K, B):
    p = wl.dense_problem(M, K, B)
    got = run(sp, p["Q"], p["scale"], p["x"])
    assert_within_bound(got, p["Q"], p["scale"], p["x"])


@pytest.mark.parametrize("q_offset,vec", [(0, 16), (4, 4), (1, 1), (2, 1)])
@pytest.mark.parametrize("M,K", [(300, 1536), (77, 64), (19, 4096)])
def test_dense_integer_inputs_bit_exact(sp, M, K, q_offset, vec):
    assert sp.dense_proj_plan(K, M, 5, q_align=q_offset or 16)["vec"] == vec
    p = wl.dense_problem(M, K, 5, seed=1, integer_x=True)
    got = run(sp, p["Q"], p["scale"], p["x"], q_offset=q_offset)
    ref = oracle.dense_forward(p["Q"], p["scale"], p["x"]).astype(np.float32)
    mism = bits32(got) != bits32(ref)
    assert not mism.any(), f"{int(mism.sum())} outputs differ, first at {np.argwhere(mism)[0]}"


@pytest.mark.parametrize("q_offset", [0, 4, 1])
def test_dense_unaligned_weights(sp, q_offset):
    p = wl.dense_problem(129, 1536, 4, seed=2)
    got = run(sp, p["Q"], p["scale"], p["x"], q_offset=q_offset)
    assert_within_bound(got, p["Q"], p["scale"], p["x"])


def test_dense_result_does_not_depend_on_batch(sp):
    """Each row's summation order depends on K only: a row computed inside a
    batch of 13 (launches of 8 + 5 rows) equals the same row computed alone."""
    p = wl.dense_problem(700, 1536, 13, seed=3)
    together = run(sp, p["Q"], p["scale"], p["x"])
    for b in range(13):
        alone = run(sp, p["Q"], p["scale"], p["x"][b:b + 1])
        np.testing.assert_array_equal(bits32(alone[0]), bits32(together[b]))


@pytest.mark.parametrize("kind", list(wl.DENSE_SHAPES))
def test_dense_model_shapes_all_outputs(sp, kind):
    """The block's continuous-input projections and the vocabulary head at
    their real sizes: every output against the oracle."""
    p = wl.dense_projection(kind, B=2)
    got = run(sp, p["Q"], p["scale"], p["x"])
    worst = assert_within_bound(got, p["Q"], p["scale"], p["x"])
    print(f"{kind}: worst error / bound = {worst:.3g}")


def test_dense_special_inputs(sp):
    """x = 0 gives 0; x = e_k gives s_m Q[m, k] exactly; a zero scale gives 0."""
    M, K = 257, 1536
    p = wl.dense_problem(M, K, 1, seed=4)
    Q, s = p["Q"], p["scale"].copy()
    x = np.zeros((3, K), dtype=np.float32)
    x[1, 5] = 1.0
    x[2, K - 1] = 1.0
    s[7] = 0.0
    got = run(sp, Q, s, x)
    np.testing.assert_array_equal(got[0], np.zeros(M, dtype=np.float32))
    np.testing.assert_array_equal(got[1], (Q[:, 5].astype(np.float32) * s))
    np.testing.assert_array_equal(got[2], (Q[:, K - 1].astype(np.float32) * s))
    assert (got[:, 7] == 0).all()


def test_dense_zero_batch_writes_nothing(sp):
    p = wl.dense_problem(40, 64, 1)
    y = torch.full((1, 40), 3.5, dtype=torch.float32, device="cuda")
    sp.dense_proj_forward(q_at(p["Q"], 0), dev(p["scale"]), dev(p["x"]), 0, y)
    torch.cuda.synchronize()
    assert (y == 3.5).all()


def test_dense_only_batch_rows_written(sp):
    """Rows b >= B of y keep their contents (a launch of 8 rows carrying 5)."""
    p = wl.dense_problem(50, 96, 8, seed=5)
    y = torch.full((8, 50), 3.5, dtype=torch.float32, device="cuda")
    sp.dense_proj_forward(q_at(p["Q"], 0), dev(p["scale"]), dev(p["x"]), 5, y)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    assert (got[5:] == 3.5).all()
    assert_within_bound(got[:5], p["Q"], p["scale"], p["x"][:5])


def test_dense_side_stream_and_graph_replay(sp):
    """Enqueued on a side stream and captured in a HIP graph: every replay
    (with other work and synchronisations between them) gives the eager result."""
    p = wl.dense_problem(1500, 1536, 2, seed=6)
    Qd, sd, xd = q_at(p["Q"], 0), dev(p["scale"]), dev(p["x"])
    y = torch.zeros((2, 1500), dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        sp.dense_proj_forward(Qd, sd, xd, 2, y, stream=side)
    side.synchronize()
    eager = y.cpu().numpy()
    assert_within_bound(eager, p["Q"], p["scale"], p["x"])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        sp.dense_proj_forward(Qd, sd, xd, 2, y, stream=side)
    for i in range(3):
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(bits32(y.cpu().numpy()), bits32(eager), err_msg=f"replay {i}")


def test_dense_rejects_bad_arguments(sp):
    p = wl.dense_problem(16, 32, 1)
    Qd, sd, xd = q_at(p["Q"], 0), dev(p["scale"]), dev(p["x"])
    y = torch.zeros((1, 16), dtype=torch.float32, device="cuda")
    with pytest.raises(sp.SpikeError, match="B = -1"):
        sp.dense_proj_forward(Qd, sd, xd, -1, y)
    xoff = torch.zeros(33, dtype=torch.float32, device="cuda")
    raw = sp.raw_library()
    rc = raw.dense_proj_forward(Qd.data_ptr(), sd.data_ptr(), 32, 16, xoff.data_ptr() + 2, 1, y.data_ptr(), None)
    assert rc == sp.SPIKE_EINVAL and "aligned" in sp.spike_proj_last_error()


@pytest.fixture
def forced_kernel(sp):
    """Set a process-wide kernel override for one test and restore it."""
    def force(kernel, wg_per_cu=0):
        sp.dense_proj_tune(sp.DENSE_TUNE_KERNEL, kernel)
        sp.dense_proj_tune(sp.DENSE_TUNE_WG_PER_CU, wg_per_cu)
    yield force
    sp.dense_proj_tune(sp.DENSE_TUNE_KERNEL, 0)
    sp.dense_proj_tune(sp.DENSE_TUNE_WG_PER_CU, 0)


# K for every register-kernel chunk count NPL = ceil(K / 512) from 1 to 8,
# with ragged tails (lanes past the row) and exact multiples.
REG_KS = [16, 496, 512, 528, 1024, 1536, 2000, 2560, 3072, 3584, 4096]


@pytest.mark.parametrize("K", REG_KS)
@pytest.mark.parametrize("B", [1, 2, 5])
@pytest.mark.parametrize("kernel", ["register", "staged"])
def test_dense_each_kernel_matches_oracle(sp, forced_kernel, K, B, kernel):
    forced_kernel(sp.DENSE_KERNEL_REGISTER if kernel == "register" else sp.DENSE_KERNEL_STAGED)
    assert sp.dense_proj_plan(K, 1031, B)["kernel"] == (
        sp.DENSE_KERNEL_REGISTER if kernel == "register" else sp.DENSE_KERNEL_STAGED)
    p = wl.dense_problem(1031, K, B, seed=7)
    got = run(sp, p["Q"], p["scale"], p["x"])
    assert_within_bound(got, p["Q"], p["scale"], p["x"])


@pytest.mark.parametrize("wg_per_cu", [1, 2, 4, 8])
def test_dense_register_kernel_many_rows_per_group(sp, forced_kernel, wg_per_cu):
    """A small grid makes each lane group walk many rows (more than 32, so the
    parked results are flushed several times, with a partial last block); an
    odd M leaves the two groups of the last wave with different row counts."""
    forced_kernel(0, wg_per_cu)
    M, K = 150001, 16
    plan = sp.dense_proj_plan(K, M, 3)
    assert plan["kernel"] == sp.DENSE_KERNEL_REGISTER and plan["workgroups"] == 256 * wg_per_cu
    p = wl.dense_problem(M, K, 3, seed=8, integer_x=True)
    got = run(sp, p["Q"], p["scale"], p["x"])
    ref = oracle.dense_forward(p["Q"], p["scale"], p["x"]).astype(np.float32)
    mism = bits32(got) != bits32(ref)
    assert not mism.any(), f"{int(mism.sum())} outputs differ, first at {np.argwhere(mism)[0]}"


def test_dense_register_kernel_grid_does_not_change_results(sp, forced_kernel):
    p = wl.dense_problem(20000, 1536, 1, seed=9)
    outs = []
    for wpc in (1, 3, 8):
        forced_kernel(0, wpc)
        outs.append(run(sp, p["Q"], p["scale"], p["x"]))
    np.testing.assert_array_equal(bits32(outs[0]), bits32(outs[1]))
    np.testing.assert_array_equal(bits32(outs[0]), bits32(outs[2]))
    assert_within_bound(outs[0], p["Q"], p["scale"], p["x"])
