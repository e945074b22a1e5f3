"""GPU parity of the INT8 quantizer/exporter (quantize.h) with the CPU oracle:
codes and scales bit for bit, in both layouts, on the model's shapes and on
edge cases (all-zero and tiny rows, binary32-created ties, huge and
subnormal magnitudes, ragged tiles, unaligned buffers), then end to end: the
exported weights drive the spike-gated and dense projections."""
from fractions import Fraction

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


def weights(M, K, seed, sigma=0.02):
    rng = np.random.default_rng([42, 13, M, K, seed])
    return rng.normal(0.0, sigma, size=(M, K)).astype(np.float32)


def at_offset(a: np.ndarray, offset: int, dtype):
    """Device copy of `a` starting `offset` bytes into a 256-byte aligned buffer."""
    nbytes = a.size * a.itemsize
    buf = torch.zeros(nbytes + 256, dtype=torch.uint8, device="cuda")
    view = buf[offset:offset + nbytes].view(dtype).view(a.shape)
    view.copy_(torch.from_numpy(np.ascontiguousarray(a)))
    return view


def gpu_quantize(sp, W, layout, w_offset=0, q_offset=0):
    M, K = W.shape
    Wd = at_offset(W, w_offset, torch.float32)
    qbuf = torch.full((M * K + 256,), 99, dtype=torch.int8, device="cuda")
    Qd = qbuf[q_offset:q_offset + M * K]
    s = torch.full((M,), float("nan"), dtype=torch.float32, device="cuda")
    sp.spike_quantize_int8(Wd, layout, Qd, s)
    torch.cuda.synchronize()
    Q = Qd.cpu().numpy()
    Q = Q.reshape(M, K) if layout == sp.SPIKE_LAYOUT_ROW_MAJOR else Q.reshape(K, M).T
    return Q, s.cpu().numpy()


def assert_same(sp, W, layout, **kw):
    Q, s = gpu_quantize(sp, W, layout, **kw)
    Qo, so = oracle.quantize_int8(W)
    np.testing.assert_array_equal(s.view(np.uint32), so.view(np.uint32))
    mism = Q != Qo
    assert not mism.any(), f"{int(mism.sum())} codes differ, first at {np.argwhere(mism)[0]}"


LAYOUTS = ["row", "col"]


def lay(sp, name):
    return sp.SPIKE_LAYOUT_ROW_MAJOR if name == "row" else sp.SPIKE_LAYOUT_COL_MAJOR


# row-major rows of K % 4 == 0 up to 4096 values take the one-pass kernel
# (every register depth: K = 4 .. 512, 1000, 1540, 2048, 4096); the others
# and every column-major case take the two-pass kernels
@pytest.mark.parametrize("M,K", [(1, 1), (5, 7), (64, 64), (65, 63), (100, 257), (128, 4), (3, 1000), (33, 1540),
                                 (7, 2048), (5, 4096), (9, 4100)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_quantizer_matches_oracle(sp, M, K, layout):
    assert_same(sp, weights(M, K, 0), lay(sp, layout))


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("w_offset,q_offset", [(4, 0), (0, 1), (8, 2)])
def test_quantizer_unaligned_buffers(sp, layout, w_offset, q_offset):
    assert_same(sp, weights(96, 200, 1), lay(sp, layout), w_offset=w_offset, q_offset=q_offset)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_quantizer_edge_rows(sp, layout):
    """All-zero and sub-floor rows, huge and subnormal magnitudes, exact ties,
    and quotients whose binary32 rounding lands on a tie."""
    W = weights(12, 80, 2)
    W[0] = 0.0
    W[1] = 0.0
    W[1, 3], W[1, 7] = 1e-9, -1e-9
    W[2] *= np.float32(1e30)
    W[3] = np.float32(1e-40) * np.sign(W[3])       # subnormal, below the floor
    W[4, :5] = [127.0, 2.5, -2.5, 3.5, 126.5]
    W[4, 5:] = 0.0
    row = 5
    for amax in (100.3, 139.1, 1.37, 201.9, 9.81, 55.5):
        amax = np.float32(amax)
        s = np.float32(amax / np.float32(127))
        for n in range(0, 126, 2):
            x = np.float32(np.float64(n + 0.5) * np.float64(s))
            if np.float32(x / s) == np.float32(n + 0.5) and Fraction(float(x)) / Fraction(float(s)) > n + 0.5:
                W[row] = 0.0
                W[row, :3] = [amax, x, -x]
                break
        row += 1
    assert_same(sp, W, lay(sp, layout))
    Q, _ = gpu_quantize(sp, W, lay(sp, layout))
    assert (Q[0] == 0).all() and (Q[1, [3, 7]] == [13, -13]).all()
    assert list(Q[4, :5]) == [127, 2, -2, 4, 126]


@pytest.mark.parametrize("kind,layout", [("tcam", "col"), ("down", "col"), ("qkvo", "row"), ("up", "row"),
                                         ("head", "row")])
def test_quantizer_model_shapes(sp, kind, layout):
    """The model's matrices as the exporter writes them: binary-input
    projections column-major, continuous-input ones row-major."""
    K, M = {"tcam": (1536, 1536), "down": (6144, 1536), **wl.DENSE_SHAPES}[kind]
    assert_same(sp, weights(M, K, 3), lay(sp, layout))


def test_exported_weights_drive_the_spike_projection(sp):
    """FFN down [1536][6144] quantized on the GPU into the column-major layout
    and run through spike_proj_forward: bit-identical to the oracle's
    projection of the oracle's own export."""
    M, K, B = 1536, 6144, 3
    W = weights(M, K, 4)
    Wd = torch.from_numpy(W).cuda()
    Qd = torch.empty((K, M), dtype=torch.int8, device="cuda")
    sd = torch.empty(M, dtype=torch.float32, device="cuda")
    sp.spike_quantize_int8(Wd, sp.SPIKE_LAYOUT_COL_MAJOR, Qd, sd)
    h = sp.spike_proj_create(Qd, sd)
    bits = np.random.default_rng(9).random((B, K)) < 0.1
    masks = wl.pack_bits(bits)
    out = torch.empty((B, M), dtype=torch.float32, device="cuda")
    sp.spike_proj_forward(h, torch.from_numpy(masks.view(np.int64)).cuda(), B, out)
    torch.cuda.synchronize()
    Qo, so = oracle.quantize_int8(W)
    ref = oracle.spike_forward(oracle.export_column_major(Qo), so, masks)
    np.testing.assert_array_equal(out.cpu().numpy().view(np.uint32), ref.view(np.uint32))
    h.close()


def test_exported_weights_drive_the_dense_projection(sp):
    """FFN up [6144][1536] quantized row-major on the GPU, then the dense
    projection: equal to the dense projection of the oracle's export."""
    M, K = 6144, 1536
    W = weights(M, K, 5)
    Wd = torch.from_numpy(W).cuda()
    Qd = torch.empty((M, K), dtype=torch.int8, device="cuda")
    sd = torch.empty(M, dtype=torch.float32, device="cuda")
    sp.spike_quantize_int8(Wd, sp.SPIKE_LAYOUT_ROW_MAJOR, Qd, sd)
    x = np.random.default_rng(10).standard_normal((2, K)).astype(np.float32)
    y = torch.empty((2, M), dtype=torch.float32, device="cuda")
    sp.dense_proj_forward(Qd, sd, torch.from_numpy(x).cuda(), 2, y)
    Qo, so = oracle.quantize_int8(W)
    np.testing.assert_array_equal(Qd.cpu().numpy(), Qo)
    y2 = torch.empty_like(y)
    sp.dense_proj_forward(torch.from_numpy(Qo).cuda(), torch.from_numpy(so).cuda(), torch.from_numpy(x).cuda(), 2, y2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy().view(np.uint32), y2.cpu().numpy().view(np.uint32))


def test_quantizer_rejects_bad_arguments(sp):
    W = torch.zeros((4, 4), dtype=torch.float32, device="cuda")
    Q = torch.zeros(16, dtype=torch.int8, device="cuda")
    s = torch.zeros(4, dtype=torch.float32, device="cuda")
    with pytest.raises(sp.SpikeError, match="layout"):
        sp.spike_quantize_int8(W, 7, Q, s)
    with pytest.raises(ValueError):
        sp.spike_quantize_int8(W, sp.SPIKE_LAYOUT_ROW_MAJOR, Q[:8], s)
