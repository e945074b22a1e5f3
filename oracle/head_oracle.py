"""Output-head candidate-row verification (TEST INFRASTRUCTURE ONLY).

Paper Sec. 5 ("Output-Head Power Case Study", projection-only trace): the
vocabulary projection runs with INT8 activations over all V rows; when the
gap between the two largest of these approximate logits is below a
threshold, the K highest-scoring rows are recomputed with the FP32
activations and the greedy token is the best of the recomputed rows;
otherwise it is the approximate top row.  This module takes the steps in
that order:

1. activations: symmetric INT8 with one scale per activation vector, the
   formulas of Sec. 2.3 applied to x (binary32, ties to even, 1e-8 floor):
       s_x = max(max_k |x_k|, 1e-8) / 127,  xq_k = clip(round(x_k / s_x), -127, 127)
2. approximate logits: the exact integer dot product acc_m = sum_k Q[m,k] xq_k,
   then fl32(fl32(acc_m) * fl32(s_m * s_x));
3. candidates: the K rows with the largest approximate logits, largest
   first, equal logits in ascending row order;
4. gate: gap = fl32(l(1) - l(2)) over the two largest approximate logits of
   all V rows (+inf when V = 1); verification runs when gap < threshold;
5. verification: each candidate row's logit recomputed with the FP32
   activations, s_m * sum_k Q[m,k] x_k, here exactly (float64); the token is
   the candidate with the largest recomputed logit (ties: the lower row).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module; the GPU library never does.
"""
from __future__ import annotations

import numpy as np

from .quant_oracle import FLOOR, QMAX


def quantize_activations(x: np.ndarray):
    """xq int8 [K] and s_x float32 for one FP32 activation vector."""
    x = np.asarray(x)
    if x.dtype != np.float32 or x.ndim != 1 or x.size < 1:
        raise ValueError("x must be a non-empty float32 vector")
    amax = np.float32(np.max(np.abs(x)))
    sx = np.float32(max(amax, FLOOR) / QMAX)
    xq = np.clip(np.rint(x / sx), -127, 127).astype(np.int8)
    return xq, sx


def approx_logits(Q: np.ndarray, scale: np.ndarray, x: np.ndarray) -> np.ndarray:
    """Step 2: float32 [V] logits of the INT8-activation head."""
    Q = np.asarray(Q, dtype=np.int8)
    scale = np.asarray(scale, dtype=np.float32)
    xq, sx = quantize_activations(x)
    acc = Q.astype(np.int64) @ xq.astype(np.int64)  # exact; |acc| <= 127 * 127 * K
    c = (scale * sx).astype(np.float32)             # binary32 products
    return (acc.astype(np.float32) * c).astype(np.float32)


def top_candidates(logits: np.ndarray, k: int) -> np.ndarray:
    """Step 3: indices of the k largest logits, largest first, ties by row."""
    logits = np.asarray(logits, dtype=np.float32)
    order = sorted(range(logits.size), key=lambda m: (-float(logits[m]), m))
    return np.array(order[:k], dtype=np.int32)


def head_verify(Q: np.ndarray, scale: np.ndarray, x: np.ndarray, k: int, threshold: float):
    """Steps 1-5.  Returns a dict: logits (approximate, float32 [V]),
    cand (int32 [k]), gap (float32), verified (bool), recomputed (float64 [k],
    or None when verification did not run) and token (int)."""
    Q = np.asarray(Q, dtype=np.int8)
    V = Q.shape[0]
    if not 1 <= k <= V:
        raise ValueError("need 1 <= k <= V")
    logits = approx_logits(Q, scale, x)
    top2 = top_candidates(logits, min(2, V))
    gap = np.float32(logits[top2[0]] - logits[top2[1]]) if V > 1 else np.float32(np.inf)
    cand = top_candidates(logits, k)
    verified = bool(gap < np.float32(threshold))
    rec = None
    token = int(cand[0])
    if verified:
        xd = np.asarray(x, dtype=np.float64)
        rec = np.array([float(scale[m]) * float(Q[m].astype(np.float64) @ xd) for m in cand])
        best = max(range(k), key=lambda i: (rec[i], -int(cand[i])))
        token = int(cand[best])
    return dict(logits=logits, cand=cand, gap=gap, verified=verified, recomputed=rec, token=token)
