"""Symmetric per-output-channel INT8 quantizer (TEST INFRASTRUCTURE ONLY).

Paper Sec. 2.3 ("Quantization and Accumulation"), for a weight matrix W of
shape [M, K] (M output channels, K inputs):

    s_m     = max(max_k |W[m, k]|, 1e-8) / 127
    Q[m, k] = clip(round(W[m, k] / s_m), -127, 127)

Arithmetic is binary32 throughout (the exporter works on FP32 weights and the
runtime stores FP32 scales): the maximum of |W| is exact, 1e-8 is its nearest
binary32 value, the two divisions are correctly rounded binary32 divisions,
and round() resolves ties to even (the reading taken for the paper's
unspecified tie rule; an exporter built on PyTorch rounds this way).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module; the GPU library never does.
"""
from __future__ import annotations

import numpy as np

FLOOR = np.float32(1e-8)
QMAX = np.float32(127)


def quantize_int8(W: np.ndarray):
    """Q int8 [M, K] (logical, row m = output channel m) and s float32 [M]."""
    W = np.asarray(W)
    if W.dtype != np.float32 or W.ndim != 2 or W.shape[0] < 1 or W.shape[1] < 1:
        raise ValueError("W must be a non-empty float32 matrix [M, K]")
    M, K = W.shape
    s = np.empty(M, dtype=np.float32)
    Q = np.empty((M, K), dtype=np.int8)
    for m in range(M):
        amax = np.float32(np.max(np.abs(W[m])))
        s[m] = np.float32(max(amax, FLOOR) / QMAX)          # binary32 division
        r = np.rint(W[m] / s[m])                             # binary32 division, ties to even
        Q[m] = np.clip(r, -127, 127).astype(np.int8)
    return Q, s


def export_column_major(Q: np.ndarray) -> np.ndarray:
    """Storage of the binary-input projections: W_cm[k, m] = Q[m, k] (Sec. 2.2)."""
    return np.ascontiguousarray(np.asarray(Q, dtype=np.int8).T)
