"""Seeded synthetic workloads for the spike-gated INT8 projection.

The inputs are shaped like the binary-input projections of the paper's
874M-parameter spiking decoder (Sec. 2.1: 22 blocks, a 1536-wide residual
stream; the TCAM projection and the feed-forward down projection take binary
inputs).  The paper releases no weights or activations (Artifact
Availability), so every array here is drawn from a seeded generator.

This module is shared by the tests, the benchmark and the oracle checks.  It
holds no arithmetic of the projection itself: it only draws weights, scales
and spike bits and packs the bits into the library's bitmask layout.

Spike bitmask layout (the library's input format): row ``b`` of a batch is
``ceil(K/64)`` little-endian 64-bit words; bit ``k`` of the row is bit
``k % 64`` of word ``k // 64``.  That is byte-for-byte
``np.packbits(bits, axis=1, bitorder="little")`` padded to 8-byte rows.

Stream seeds: every (workload, layer, projection, purpose) gets its own
generator ``np.random.default_rng([42, workload, layer, proj, purpose])``, so
any piece can be regenerated on its own and a shorter run draws a prefix of a
longer one.  42 is the decode seed the paper uses (Sec. 3.1).
"""
from __future__ import annotations

import numpy as np

SEED = 42
RESIDUAL = 1536          # residual width (Sec. 2.1)
FFN_HIDDEN = 4 * RESIDUAL  # input width of the FFN down projection (App. A.2)
N_BLOCKS = 22            # decoder blocks (Sec. 2.1)

# Projection kinds of one block, in the order a block runs them.
PROJ_TCAM = 0            # spike-conditioned TCAM projection, 1536 -> 1536
PROJ_DOWN = 1            # FFN down projection, 6144 -> 1536
PROJ_SHAPES = {PROJ_TCAM: (RESIDUAL, RESIDUAL), PROJ_DOWN: (FFN_HIDDEN, RESIDUAL)}  # (K, N)

# Purposes (last seed word) so that streams never overlap.
_P_W, _P_SCALE, _P_MASK, _P_RATE, _P_HOT, _P_ROWRATE = 0, 1, 2, 3, 4, 5

# Workload ids (first seed word after 42).
W_SINGLE, W_DOWN_SWEEP, W_STACK, W_PREFILL, W_BATCHED_STACK, W_DENSE, W_TESTS = 1, 2, 3, 4, 5, 6, 9

# Continuous-input projections of one block and the head (Sec. 2.1): row-major
# INT8 weights [M, K] applied to FP32 activations.  (K, M) per kind.
VOCAB = 57344            # output vocabulary slots of the deployed model (Sec. 2.1)
DENSE_SHAPES = {
    "qkvo": (RESIDUAL, RESIDUAL),      # attention query/key/value/output, 1536 -> 1536
    "up": (RESIDUAL, FFN_HIDDEN),      # FFN up projection, 1536 -> 6144
    "head": (RESIDUAL, VOCAB),         # vocabulary output projection, 1536 -> 57344
}

DOWN_SWEEP_RATES = (0.02, 0.05, 0.10, 0.20, 0.40)


def rng_for(workload: int, layer: int, proj: int, purpose: int) -> np.random.Generator:
    return np.random.default_rng([SEED, workload, layer, proj, purpose])


def words_per_row(K: int) -> int:
    return (int(K) + 63) // 64


def pack_bits(bits: np.ndarray) -> np.ndarray:
    """bool/0-1 array [B, K] -> uint64 bitmask [B, ceil(K/64)] (LSB-first)."""
    bits = np.asarray(bits)
    if bits.ndim != 2:
        raise ValueError("bits must be 2-D [B, K]")
    B, K = bits.shape
    nw = words_per_row(K)
    packed = np.packbits(bits.astype(bool), axis=1, bitorder="little")
    rows = np.zeros((B, nw * 8), dtype=np.uint8)
    rows[:, : packed.shape[1]] = packed
    return rows.view("<u8").reshape(B, nw)


def unpack_bits(mask: np.ndarray, K: int) -> np.ndarray:
    """uint64 bitmask [B, ceil(K/64)] -> bool [B, K] (padding bits dropped)."""
    mask = np.ascontiguousarray(mask, dtype="<u8")
    B = mask.shape[0]
    by = mask.view(np.uint8).reshape(B, -1)
    return np.unpackbits(by, axis=1, bitorder="little")[:, :K].astype(bool)


# ----------------------------------------------------------------------------
# Weight and scale draws
# ----------------------------------------------------------------------------

def uniform_weights(rng: np.random.Generator, K: int, N: int) -> np.ndarray:
    """INT8 weights uniform on [-127, 127], stored column-major: array [K, N],
    so column k of the logical [N, K] matrix is the contiguous row W[k]."""
    return rng.integers(-127, 127, size=(K, N), dtype=np.int8, endpoint=True)


def gaussian_weights(rng: np.random.Generator, K: int, N: int, sigma: float = 30.0) -> np.ndarray:
    """INT8 weights ~ N(0, sigma) rounded to nearest and clipped to [-127, 127]."""
    w = np.rint(rng.normal(0.0, sigma, size=(K, N)))
    return np.clip(w, -127, 127).astype(np.int8)


def uniform_scales(rng: np.random.Generator, N: int, lo: float = 1e-3, hi: float = 1e-2) -> np.ndarray:
    return rng.uniform(lo, hi, N).astype(np.float32)


def bernoulli_bits(rng: np.random.Generator, B: int, K: int, p: float) -> np.ndarray:
    return rng.random((B, K)) < p


# ----------------------------------------------------------------------------
# The five workloads
# ----------------------------------------------------------------------------

def single_projection(n_masks: int = 1, p: float = 0.10, K: int = RESIDUAL, N: int = RESIDUAL):
    """One 1536 -> 1536 projection at batch 1, i.i.d. Bernoulli(0.10) spikes.

    Returns dict(W [K,N] int8, scale [N] f32, masks [n_masks, words] u64, K, N).
    Each mask row is one independent batch-1 call.
    """
    W = uniform_weights(rng_for(W_SINGLE, 0, 0, _P_W), K, N)
    s = uniform_scales(rng_for(W_SINGLE, 0, 0, _P_SCALE), N)
    bits = bernoulli_bits(rng_for(W_SINGLE, 0, 0, _P_MASK), n_masks, K, p)
    return dict(W=W, scale=s, masks=pack_bits(bits), K=K, N=N, p=p)


def down_sweep(p: float, n_masks: int = 1, K: int = FFN_HIDDEN, N: int = RESIDUAL):
    """FFN down projection 6144 -> 1536 at batch 1, i.i.d. Bernoulli(p) spikes,
    p one of DOWN_SWEEP_RATES.  W and scale are shared by all rates."""
    if p not in DOWN_SWEEP_RATES:
        raise ValueError(f"rate {p} not in {DOWN_SWEEP_RATES}")
    W = uniform_weights(rng_for(W_DOWN_SWEEP, 0, 0, _P_W), K, N)
    s = uniform_scales(rng_for(W_DOWN_SWEEP, 0, 0, _P_SCALE), N)
    pi = DOWN_SWEEP_RATES.index(p)
    bits = bernoulli_bits(rng_for(W_DOWN_SWEEP, pi, 0, _P_MASK), n_masks, K, p)
    return dict(W=W, scale=s, masks=pack_bits(bits), K=K, N=N, p=p)


def stack_layer_rates(n_layers: int = N_BLOCKS) -> np.ndarray:
    """Per-block spike rate r_l ~ U[0.05, 0.20], shared by both projections of
    the block and fixed across tokens."""
    return rng_for(W_STACK, 0, 0, _P_RATE).uniform(0.05, 0.20, n_layers)


def stack_projection(layer: int, proj: int):
    """Weights and scales of one projection of the 22-block decode stack."""
    K, N = PROJ_SHAPES[proj]
    W = uniform_weights(rng_for(W_STACK, layer, proj, _P_W), K, N)
    s = uniform_scales(rng_for(W_STACK, layer, proj, _P_SCALE), N)
    return W, s


def stack_masks(layer: int, proj: int, n_tokens: int, rates: np.ndarray | None = None) -> np.ndarray:
    """Fresh Bernoulli(r_l) spikes for each of n_tokens tokens: u64 [T, words]."""
    if rates is None:
        rates = stack_layer_rates()
    K, _ = PROJ_SHAPES[proj]
    bits = bernoulli_bits(rng_for(W_STACK, layer, proj, _P_MASK), n_tokens, K, float(rates[layer]))
    return pack_bits(bits)


def stack_order(n_layers: int = N_BLOCKS):
    """(layer, proj) pairs in execution order: per block, TCAM then down."""
    return [(l, j) for l in range(n_layers) for j in (PROJ_TCAM, PROJ_DOWN)]


def stack_token_masks(n_tokens: int, n_layers: int = N_BLOCKS) -> np.ndarray:
    """All spike masks of the decode stack in stream layout: for each token,
    the masks of its projections in execution order, concatenated.  Returns
    u64 [n_tokens, sum_j words_j]."""
    rates = stack_layer_rates()
    parts = [stack_masks(l, j, n_tokens, rates) for (l, j) in stack_order(n_layers)]
    return np.ascontiguousarray(np.concatenate(parts, axis=1))


def prefill_bits(B: int = 512, K: int = FFN_HIDDEN, p: float = 0.10, stay: float = 0.5) -> np.ndarray:
    """Temporally correlated spikes for a B-token prefill of the down projection.

    Each neuron is a two-state Markov chain over the token index: x_0 ~
    Bernoulli(p); an active neuron stays active with probability `stay`; an
    inactive one turns on with probability q = p (1 - stay) / (1 - p), which
    makes p the stationary firing rate (q = 1/18 for p = 0.1, stay = 0.5).
    Returns bool [B, K].
    """
    rng = rng_for(W_PREFILL, 0, 0, _P_MASK)
    q = p * (1.0 - stay) / (1.0 - p)
    u = rng.random((B, K))
    x = np.empty((B, K), dtype=bool)
    x[0] = u[0] < p
    for t in range(1, B):
        x[t] = np.where(x[t - 1], u[t] < stay, u[t] < q)
    return x


def prefill_projection(B: int = 512, K: int = FFN_HIDDEN, N: int = RESIDUAL):
    W = uniform_weights(rng_for(W_PREFILL, 0, 0, _P_W), K, N)
    s = uniform_scales(rng_for(W_PREFILL, 0, 0, _P_SCALE), N)
    return dict(W=W, scale=s, masks=pack_bits(prefill_bits(B, K)), K=K, N=N)


def batched_stack_projection(layer: int, proj: int):
    """Weights (N(0,30) clipped) and scales of one projection of the batched
    decode stack."""
    K, N = PROJ_SHAPES[proj]
    W = gaussian_weights(rng_for(W_BATCHED_STACK, layer, proj, _P_W), K, N)
    s = uniform_scales(rng_for(W_BATCHED_STACK, layer, proj, _P_SCALE), N)
    return W, s


def batched_stack_bits(layer: int, proj: int, B: int = 64, n_steps: int = 16,
                       hot_frac: float = 0.05, hot_p: float = 0.9) -> np.ndarray:
    """Structured spikes for B sequences over n_steps decode steps.

    A fixed 'hot' set of round(hot_frac*K) columns fires with probability
    hot_p; every other column of row b fires with a per-row rate
    p_b ~ Beta(2, 18) (mean 0.10), fixed across steps.  Returns bool
    [n_steps, B, K].
    """
    K, _ = PROJ_SHAPES[proj]
    hot = rng_for(W_BATCHED_STACK, layer, proj, _P_HOT).choice(K, size=int(round(hot_frac * K)), replace=False)
    p_row = rng_for(W_BATCHED_STACK, layer, proj, _P_ROWRATE).beta(2.0, 18.0, B)
    prob = np.repeat(p_row[:, None], K, axis=1)
    prob[:, hot] = hot_p
    u = rng_for(W_BATCHED_STACK, layer, proj, _P_MASK).random((n_steps, B, K))
    return u < prob[None]


def dense_projection(kind: str, B: int = 1):
    """Row-major INT8 weights Q [M, K] ~ rounded N(0, 30), scales on
    [1e-3, 1e-2] and FP32 activations x [B, K] ~ N(0, 1) (the scale of a
    layer-normalised residual stream) for one continuous-input projection."""
    K, M = DENSE_SHAPES[kind]
    proj = list(DENSE_SHAPES).index(kind)
    Q = gaussian_weights(rng_for(W_DENSE, 0, proj, _P_W), M, K)
    s = uniform_scales(rng_for(W_DENSE, 0, proj, _P_SCALE), M)
    x = rng_for(W_DENSE, 0, proj, _P_MASK).standard_normal((B, K)).astype(np.float32)
    return dict(Q=Q, scale=s, x=x, K=K, M=M, B=B)


def dense_problem(M: int, K: int, B: int, seed: int = 0, integer_x: bool = False):
    """Small seeded dense problem of any shape.  integer_x draws x from the
    integers in [-8, 8], so that every partial sum of |Q x| stays an exact
    FP32 integer for K up to 16,512."""
    rng = np.random.default_rng([SEED, W_TESTS, 1, M, K, B, seed])
    Q = rng.integers(-127, 127, size=(M, K), dtype=np.int8, endpoint=True)
    s = uniform_scales(rng, M)
    if integer_x:
        x = rng.integers(-8, 8, size=(B, K), endpoint=True).astype(np.float32)
    else:
        x = rng.standard_normal((B, K)).astype(np.float32)
    return dict(Q=Q, scale=s, x=x, K=K, M=M, B=B)


def small_problem(K: int, N: int, B: int, p: float, seed: int = 0, w_lo: int = -127, w_hi: int = 127):
    """Small seeded problem of any shape for parity and edge-case tests."""
    rng = np.random.default_rng([SEED, W_TESTS, K, N, B, seed])
    W = rng.integers(w_lo, w_hi, size=(K, N), dtype=np.int8, endpoint=True)
    s = uniform_scales(rng, N)
    bits = rng.random((B, K)) < p
    return dict(W=W, scale=s, masks=pack_bits(bits), bits=bits, K=K, N=N, B=B)
