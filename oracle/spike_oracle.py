"""ctypes loader for the plain C oracle in spike_oracle.c.

TEST INFRASTRUCTURE ONLY: it lets the tests, the smoke check and the
benchmark's CPU baseline call the oracle on numpy arrays.  The oracle follows
the paper's Sec. 2.2-2.3 (Eq. (sparse)): active index set, INT32 sum of the
active columns, one FP32 conversion and one FP32 scale multiply per output
channel.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spike_oracle.c")
_LIB = os.path.join(_HERE, "libspike_oracle.so")
_lib = None

# No fast-math and no contraction: the epilogue must be one binary32 multiply.
CFLAGS = ["-std=c11", "-O2", "-fPIC", "-shared", "-pthread", "-ffp-contract=off",
          "-fno-fast-math", "-Wall", "-Wextra", "-Werror"]


def build(force: bool = True) -> str:
    """Compile spike_oracle.c into libspike_oracle.so next to it."""
    global _lib
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp], check=True)
        os.replace(tmp, _LIB)
        _lib = None
    return _LIB


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        p, i64 = ctypes.c_void_p, ctypes.c_int64
        lib.oracle_active_indices.argtypes = [p, i64, p]
        lib.oracle_active_indices.restype = i64
        lib.oracle_spike_acc.argtypes = [p, i64, i64, p, i64, p]
        lib.oracle_spike_acc.restype = ctypes.c_int
        lib.oracle_spike_forward.argtypes = [p, p, i64, i64, p, i64, p, ctypes.c_int]
        lib.oracle_spike_forward.restype = ctypes.c_int
        lib.oracle_dense_forward.argtypes = [p, p, i64, i64, p, i64, p]
        lib.oracle_dense_forward.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _mask2d(mask: np.ndarray, K: int) -> np.ndarray:
    mask = np.ascontiguousarray(mask, dtype=np.uint64)
    if mask.ndim == 1:
        mask = mask[None]
    if mask.shape[1] != (K + 63) // 64:
        raise ValueError(f"mask rows must hold ceil(K/64) = {(K + 63) // 64} words, got {mask.shape[1]}")
    return mask


def active_indices(mask_row: np.ndarray, K: int) -> np.ndarray:
    """Ascending active indices {k : x_k = 1} of one packed spike row."""
    row = _mask2d(mask_row, K)[0]
    idx = np.empty(max(K, 1), dtype=np.int32)
    n = load().oracle_active_indices(_ptr(row), K, _ptr(idx))
    return idx[:n].copy()


def spike_acc(W: np.ndarray, mask: np.ndarray) -> np.ndarray:
    """INT32 accumulators [B, N] for column-major INT8 W [K, N]."""
    W = np.ascontiguousarray(W, dtype=np.int8)
    K, N = W.shape
    mask = _mask2d(mask, K)
    B = mask.shape[0]
    acc = np.empty((B, N), dtype=np.int32)
    rc = load().oracle_spike_acc(_ptr(W), K, N, _ptr(mask), B, _ptr(acc))
    if rc != 0:
        raise RuntimeError(f"oracle_spike_acc failed ({rc})")
    return acc


def spike_forward(W: np.ndarray, scale: np.ndarray, mask: np.ndarray, threads: int = 1) -> np.ndarray:
    """FP32 outputs [B, N] = fl32(fl32(acc) * scale[n])."""
    W = np.ascontiguousarray(W, dtype=np.int8)
    K, N = W.shape
    scale = np.ascontiguousarray(scale, dtype=np.float32)
    if scale.shape != (N,):
        raise ValueError(f"scale must have one entry per output channel ({N}), got {scale.shape}")
    mask = _mask2d(mask, K)
    B = mask.shape[0]
    out = np.empty((B, N), dtype=np.float32)
    rc = load().oracle_spike_forward(_ptr(W), _ptr(scale), K, N, _ptr(mask), B, _ptr(out), int(threads))
    if rc != 0:
        raise RuntimeError(f"oracle_spike_forward failed ({rc})")
    return out


def dense_forward(Q: np.ndarray, scale: np.ndarray, x: np.ndarray) -> np.ndarray:
    """Dense continuous-input projection, float64 [B, M]: y = scale[m] * sum_k Q[m, k] * x[b, k]
    for row-major INT8 Q [M, K], FP32 scale [M] and FP32 x [B, K]."""
    Q = np.ascontiguousarray(Q, dtype=np.int8)
    M, K = Q.shape
    scale = np.ascontiguousarray(scale, dtype=np.float32)
    if scale.shape != (M,):
        raise ValueError(f"scale must have one entry per output channel ({M}), got {scale.shape}")
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None]
    if x.shape[1] != K:
        raise ValueError(f"x rows must hold K = {K} values, got {x.shape[1]}")
    y = np.empty((x.shape[0], M), dtype=np.float64)
    rc = load().oracle_dense_forward(_ptr(Q), _ptr(scale), K, M, _ptr(x), x.shape[0], _ptr(y))
    if rc != 0:
        raise RuntimeError(f"oracle_dense_forward failed ({rc})")
    return y
