"""GPU parity of the output-head candidate verification (head_verify.h) with
the CPU oracle.

Exact parts (bit for bit): the approximate logits, the candidate rows and
their order, the gap and the gate decision, and the approximate candidate
logits when verification does not run.  FP32 part: the verified candidate
logits, within the bound of the kernel's summation order (the dense register
kernel's: a per-lane FMA chain of at most 16 ceil(K/512) products, a 5-level
lane tree, one multiply): with u = 2^-24, gamma(n) = n u / (1 - n u) and
h = 16 ceil(K/512) + 6 (one slack level),
|rec - exact| <= u |exact| + (1 + u) s_m gamma(h) sum_k |Q x|;
and bit for bit dense_proj_forward's outputs for the candidate rows.
The token is then the oracle's unless the oracle's best recomputed logits
lie within twice that bound of each other, where any of the near-tied rows
is a correct answer.
"""
import numpy as np
import pytest
import torch

from oracle import head_oracle
from paper_2606_03026_amd import workloads as wl
from tests.golden.load import load_head_example

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(scope="module")
def sp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_03026_amd import _binding
    return _binding


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_head(sp, Q, s, x, k, thr, Qd=None):
    V = Q.shape[0]
    logits = torch.full((V,), float("nan"), dtype=torch.float32, device="cuda")
    cand = torch.full((k,), -1, dtype=torch.int32, device="cuda")
    cl = torch.full((k,), float("nan"), dtype=torch.float32, device="cuda")
    res = torch.full((2,), -1, dtype=torch.int32, device="cuda")
    sp.head_verify_forward(dev(Q) if Qd is None else Qd, dev(s), dev(x), k, thr, logits, cand, cl, res)
    torch.cuda.synchronize()
    return dict(logits=logits.cpu().numpy(), cand=cand.cpu().numpy(), cand_logits=cl.cpu().numpy(),
                token=int(res[0]), verified=bool(res[1]))


def rec_bound(Q, s, x, rows):
    K = Q.shape[1]
    h = 16 * (-(-K // 512)) + 6
    gamma = h * U / (1 - h * U)
    absdot = np.abs(Q[rows].astype(np.float64)) @ np.abs(x.astype(np.float64))
    exact = s[rows].astype(np.float64) * (Q[rows].astype(np.float64) @ x.astype(np.float64))
    return U * np.abs(exact) + (1 + U) * s[rows].astype(np.float64) * gamma * absdot


def assert_head_parity(got, Q, s, x, k, thr):
    ref = head_oracle.head_verify(Q, s, x, k, thr)
    np.testing.assert_array_equal(got["logits"].view(np.uint32), ref["logits"].view(np.uint32))
    np.testing.assert_array_equal(got["cand"], ref["cand"])
    assert got["verified"] == ref["verified"], (ref["gap"], thr)
    c = ref["cand"]
    if not ref["verified"]:
        np.testing.assert_array_equal(got["cand_logits"].view(np.uint32), ref["logits"][c].view(np.uint32))
        assert got["token"] == int(c[0])
        return ref
    lim = rec_bound(Q, s, x, c)
    err = np.abs(got["cand_logits"].astype(np.float64) - ref["recomputed"])
    assert (err <= lim).all(), f"recomputed logits outside the bound: {err.max():.3e}"
    rec = ref["recomputed"]
    order = sorted(range(k), key=lambda i: (-rec[i], int(c[i])))
    near = {int(c[i]) for i in order if rec[order[0]] - rec[i] <= 2 * (lim[order[0]] + lim[i])}
    if len(near) == 1:
        assert got["token"] == ref["token"]
    else:
        assert got["token"] in near
    return ref


def head_problem(V, K, seed):
    rng = np.random.default_rng([42, 16, V, K, seed])
    Q = np.clip(np.rint(rng.normal(0, 30, size=(V, K))), -127, 127).astype(np.int8)
    s = rng.uniform(1e-3, 1e-2, V).astype(np.float32)
    x = rng.standard_normal(K).astype(np.float32)
    return Q, s, x


def test_hand_example_padded_to_16_inputs(sp):
    g = load_head_example()
    K = 16
    Q = np.zeros((g["V"], K), dtype=np.int8)
    Q[:, :g["K"]] = g["Q"]
    x = np.zeros(K, dtype=np.float32)
    x[:g["K"]] = g["x"]
    for k, thr, verified, token in g["case"]:
        got = gpu_head(sp, Q, g["scale"], x, k, thr)
        np.testing.assert_array_equal(got["logits"], g["logits"].astype(np.float32))
        assert (got["verified"], got["token"]) == (verified, token)
        assert list(got["cand"]) == list(g["order"][:k])


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("k", [16, 32, 64])
@pytest.mark.parametrize("thr", [0.5, 4.0])
def test_vocabulary_head(sp, seed, k, thr):
    """The 1536 -> 57,344 head with the paper's K and gate thresholds."""
    d = wl.dense_projection("head", B=1)
    x = np.random.default_rng([42, 17, seed]).standard_normal(1536).astype(np.float32)
    got = gpu_head(sp, d["Q"], d["scale"], x, k, thr)
    assert_head_parity(got, d["Q"], d["scale"], x, k, thr)


@pytest.mark.parametrize("V,K", [(1, 16), (2, 16), (3, 48), (63, 512), (64, 528), (65, 1536), (1000, 4096),
                                 (4097, 96), (20000, 1536)])
@pytest.mark.parametrize("k", [1, 2, 64])
@pytest.mark.parametrize("thr", [0.0, 0.5, float("inf")])
def test_shapes_and_gate_limits(sp, V, K, k, thr):
    k = min(k, V)
    Q, s, x = head_problem(V, K, 0)
    got = gpu_head(sp, Q, s, x, k, thr)
    ref = assert_head_parity(got, Q, s, x, k, thr)
    if thr == 0.0 or V == 1:
        assert not ref["verified"]
    if thr == float("inf") and V >= 2:
        assert ref["verified"]


def test_exact_ties_take_lower_rows(sp):
    """Rows repeated in blocks give equal logits: candidates must take the
    lower rows of each tie first; an all-zero head ties everywhere."""
    base, _, x = head_problem(40, 64, 1)
    Q = np.repeat(base, 7, axis=0)               # 280 rows, 7 copies of each
    s = np.full(280, 0.004, dtype=np.float32)
    for k in (1, 5, 64):
        got = gpu_head(sp, Q, s, x, k, 0.5)
        assert_head_parity(got, Q, s, x, k, 0.5)
    Z = np.zeros((3000, 32), dtype=np.int8)
    got = gpu_head(sp, Z, np.ones(3000, dtype=np.float32), x[:32], 64, 0.5)
    assert list(got["cand"]) == list(range(64)) and got["verified"] and got["token"] == 0


@pytest.mark.parametrize("step", [13, 40])
def test_ties_across_selecting_workgroups(sp, step):
    """Rows every `step`-th of 20,000 hold the same largest logit: 1,539 tied
    rows overflow the pools (radix select over the whole array), 500 tied rows
    spread over the five selecting workgroups are merged and ranked."""
    V, K = 20000, 32
    rng = np.random.default_rng([42, 18, step])
    Q = rng.integers(-3, 4, size=(V, K)).astype(np.int8)
    Q[::step] = 100
    s = np.full(V, 0.003, dtype=np.float32)
    x = np.abs(rng.standard_normal(K)).astype(np.float32) + 0.5
    for k, thr in ((64, 0.5), (3, float("inf")), (1, 0.0)):
        got = gpu_head(sp, Q, s, x, k, thr)
        ref = assert_head_parity(got, Q, s, x, k, thr)
        assert list(ref["cand"]) == list(range(0, step * k, step))


def dense_head_rows(sp, Q, s, x):
    """dense_proj_forward over all rows of Q for the one activation vector x."""
    V, K = Q.shape
    y = torch.full((1, V), float("nan"), dtype=torch.float32, device="cuda")
    sp.dense_proj_forward(dev(Q), dev(s), dev(x.reshape(1, K)), 1, y)
    torch.cuda.synchronize()
    return y[0].cpu().numpy()


@pytest.mark.parametrize("V,K", [(57344, 1536), (20000, 1536), (1000, 4096), (3000, 2560), (4097, 96), (65, 1536),
                                 (3, 48)])
@pytest.mark.parametrize("k", [2, 16, 64])
def test_verified_logits_are_the_dense_heads(sp, V, K, k):
    """The verified candidates' logits are bit for bit the dense register
    kernel's outputs for those rows (same FMA order), whether they come from
    the lists or, after a whole-array selection, from the selection's own
    recompute (ties force that path in the second half)."""
    k = min(k, V)
    if (V, K) == (57344, 1536):
        d = wl.dense_projection("head", B=1)
        Q, s = d["Q"], d["scale"]
        x = np.random.default_rng([42, 19, k]).standard_normal(K).astype(np.float32)
    else:
        Q, s, x = head_problem(V, K, 7 + k)
    y = dense_head_rows(sp, Q, s, x)
    got = gpu_head(sp, Q, s, x, k, float("inf"))
    assert got["verified"] == (V >= 2)
    if got["verified"]:
        np.testing.assert_array_equal(got["cand_logits"].view(np.uint32), y[got["cand"]].view(np.uint32))
    assert_head_parity(got, Q, s, x, k, float("inf"))
    if V >= 200:
        Qt = Q.copy()
        Qt[::13] = 100  # many equal approximate logits: the lists cannot decide
        st = np.full(V, 0.003, dtype=np.float32)
        xt = np.abs(x) + 0.5
        yt = dense_head_rows(sp, Qt, st, xt)
        got = gpu_head(sp, Qt, st, xt, k, float("inf"))
        np.testing.assert_array_equal(got["cand_logits"].view(np.uint32), yt[got["cand"]].view(np.uint32))
        assert_head_parity(got, Qt, st, xt, k, float("inf"))
        assert list(got["cand"]) == list(range(0, 13 * k, 13))


def test_workspace_shared_by_calls(sp):
    """One explicit workspace, filled with junk first, through calls of
    different sizes, gates and selection paths on one stream."""
    ws = sp.head_verify_workspace()
    ws.fill_(0xA5)
    d = wl.dense_projection("head", B=1)
    x = np.random.default_rng(9).standard_normal(1536).astype(np.float32)
    Qt, st_, _ = head_problem(20000, 256, 5)
    cases = [(d["Q"], d["scale"], x, 64, float("inf")), (np.zeros((3000, 32), dtype=np.int8),
             np.ones(3000, dtype=np.float32), x[:32], 8, 0.5), (Qt, st_, x[:256], 16, 4.0),
             (d["Q"][:1], d["scale"][:1], x, 1, 0.5), (d["Q"], d["scale"], x, 2, 0.0)]
    for Q, s, xx, k, thr in cases:
        V = Q.shape[0]
        logits = torch.empty(V, device="cuda")
        cand = torch.empty(k, dtype=torch.int32, device="cuda")
        cl = torch.empty(k, device="cuda")
        res = torch.empty(2, dtype=torch.int32, device="cuda")
        sp.head_verify_forward(dev(Q), dev(s), dev(xx), k, thr, logits, cand, cl, res, workspace=ws)
        torch.cuda.synchronize()
        got = dict(logits=logits.cpu().numpy(), cand=cand.cpu().numpy(), cand_logits=cl.cpu().numpy(),
                   token=int(res[0]), verified=bool(res[1]))
        assert_head_parity(got, Q, s, xx, k, thr)



def test_negative_and_mixed_logits(sp):
    Q, s, x = head_problem(5000, 256, 2)
    Q[:2500] = -np.abs(Q[:2500])
    x = np.abs(x)                                 # half the logits negative
    for thr in (0.5, float("inf")):
        assert_head_parity(gpu_head(sp, Q, s, x, 64, thr), Q, s, x, 64, thr)
    Qn = -np.abs(Q)                               # every logit negative or zero
    assert_head_parity(gpu_head(sp, Qn, s, x, 16, 4.0), Qn, s, x, 16, 4.0)


def test_graph_replay_matches_eager(sp):
    d = wl.dense_projection("head", B=1)
    x = np.random.default_rng(7).standard_normal(1536).astype(np.float32)
    Qd, sd, xd = dev(d["Q"]), dev(d["scale"]), dev(x)
    V = d["Q"].shape[0]
    logits = torch.zeros(V, dtype=torch.float32, device="cuda")
    cand = torch.zeros(32, dtype=torch.int32, device="cuda")
    cl = torch.zeros(32, dtype=torch.float32, device="cuda")
    res = torch.zeros(2, dtype=torch.int32, device="cuda")
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        sp.head_verify_forward(Qd, sd, xd, 32, float("inf"), logits, cand, cl, res, stream=st)
    st.synchronize()
    eager = [t.cpu().numpy().copy() for t in (logits, cand, cl, res)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=st):
        sp.head_verify_forward(Qd, sd, xd, 32, float("inf"), logits, cand, cl, res, stream=st)
    for i in range(3):
        for t in (logits, cl):
            t.fill_(float("nan"))
        cand.fill_(-1)
        res.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(eager, (logits, cand, cl, res)):
            np.testing.assert_array_equal(a.view(np.uint32) if a.dtype == np.float32 else a,
                                          b.cpu().numpy().view(np.uint32) if a.dtype == np.float32 else b.cpu().numpy(),
                                          err_msg=f"replay {i}")


def test_rejects_bad_arguments(sp):
    Q, s, x = head_problem(10, 32, 3)
    t = [torch.zeros(10, device="cuda"), torch.zeros(16, dtype=torch.int32, device="cuda"),
         torch.zeros(16, device="cuda"), torch.zeros(2, dtype=torch.int32, device="cuda")]
    with pytest.raises(sp.SpikeError, match="top_k"):
        sp.head_verify_forward(dev(Q), dev(s), dev(x), 11, 0.5, *t)
    with pytest.raises(sp.SpikeError, match="NaN"):
        sp.head_verify_forward(dev(Q), dev(s), dev(x), 4, float("nan"), *t)
