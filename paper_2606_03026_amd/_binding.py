"""ctypes binding of libspike_proj.so (C ABI in include/spike_proj.h,
include/dense_proj.h, include/quantize.h and include/head_verify.h).

Argument marshalling only: every step of the projection runs in the HIP
kernels of the library.  Tensors are torch device tensors; their data
pointers are passed straight through.  There is no fallback: if the library
is missing, importing this module fails.
"""
from __future__ import annotations

import ctypes
import os

import torch

from .build import LIB

SPIKE_OK, SPIKE_EINVAL, SPIKE_EHIP, SPIKE_ENOMEM, SPIKE_EUNSUPPORTED = 0, -1, -2, -3, -4
SPIKE_TUNE_PATH, SPIKE_TUNE_SLICE_WORDS, SPIKE_TUNE_MFMA_MIN_B, SPIKE_TUNE_VEC, SPIKE_TUNE_MAX_SLICES = 1, 2, 3, 4, 5
SPIKE_TUNE_SHAPE, SPIKE_TUNE_TILES_PER_UNIT, SPIKE_TUNE_XCD_SPREAD, SPIKE_TUNE_MFMA_WAVES = 6, 7, 8, 9
SPIKE_TUNE_MFMA_DEPTH, SPIKE_TUNE_MFMA_ROW_TILE, SPIKE_TUNE_MFMA_COL_SETS = 11, 12, 13
SPIKE_SHAPE_NT = 1 << 25
SPIKE_SHAPE_I16 = 1 << 26
SPIKE_PATH_AUTO, SPIKE_PATH_GATHER, SPIKE_PATH_MFMA = 0, 1, 2
SPIKE_DEFAULT_MAX_B = 512
DENSE_MAX_K, DENSE_MAX_B = 16128, 65535
DENSE_KERNEL_STAGED, DENSE_KERNEL_REGISTER = 1, 2
DENSE_TUNE_KERNEL, DENSE_TUNE_WG_PER_CU = 1, 2
SPIKE_LAYOUT_ROW_MAJOR, SPIKE_LAYOUT_COL_MAJOR = 0, 1


def SPIKE_SHAPE(V: int, LG: int, U: int, BLOCK: int, NT: bool = False, I16: bool = False) -> int:
    """Shape code of the gather launch (same packing as the header macros)."""
    return (V | (LG << 5) | (U << 15) | ((BLOCK // 64) << 20) | (SPIKE_SHAPE_NT if NT else 0)
            | (SPIKE_SHAPE_I16 if I16 else 0))

EXPORTED = (
    "spike_proj_create", "spike_proj_reserve", "spike_proj_forward", "spike_proj_forward_acc",
    "spike_proj_destroy", "spike_proj_tune", "spike_compact", "spike_stack_forward",
    "spike_stream_create", "spike_stream_forward", "spike_stream_tune", "spike_stream_destroy",
    "spike_proj_last_error", "spike_proj_shapes", "spike_mfma_plans", "spike_proj_plan_query",
    "spike_proj_abi_version", "spike_proj_forward_noalloc", "spike_proj_create_reserved",
    "spike_stack_forward_fused", "dense_proj_forward", "dense_proj_plan", "dense_proj_tune",
    "spike_quantize_int8", "spike_check_scale_shape", "head_verify_forward", "head_verify_workspace_bytes",
)

if not os.path.exists(LIB):
    raise ImportError(f"{LIB} is not built; run __graft_entry__.build() (python -m paper_2606_03026_amd.build)")

_lib = ctypes.CDLL(LIB)
_p, _i32 = ctypes.c_void_p, ctypes.c_int32
_sig = {
    "spike_proj_create": [_p, _p, _i32, _i32, ctypes.POINTER(_p)],
    "spike_proj_create_reserved": [_p, _p, _i32, _i32, _i32, _i32, ctypes.POINTER(_p)],
    "spike_proj_reserve": [_p, _i32],
    "spike_proj_forward": [_p, _p, _i32, _p, _p],
    "spike_proj_forward_acc": [_p, _p, _i32, _p, _p],
    "spike_proj_forward_noalloc": [_p, _p, _i32, _i32, _p, _i32, _p, _p],
    "spike_proj_destroy": [_p],
    "spike_proj_tune": [_p, _i32, _i32],
    "spike_compact": [_p, _i32, _i32, _p, _p, _p],
    "spike_stack_forward": [_p, _i32, _p, _i32, _p, _p],
    "spike_stack_forward_fused": [_p, _i32, _p, _i32, _p, _p],
    "spike_stream_create": [_p, _i32, _i32, _i32, ctypes.POINTER(_p)],
    "spike_stream_forward": [_p, _p, _p, _p],
    "spike_stream_tune": [_p, _i32, _i32],
    "spike_stream_destroy": [_p],
    "spike_proj_abi_version": [],
    "spike_proj_shapes": [_p, _i32],
    "spike_mfma_plans": [_p, _i32],
    "spike_proj_plan_query": [_i32, _i32, _i32, _p, _p],
    "dense_proj_forward": [_p, _p, _i32, _i32, _p, _i32, _p, _p],
    "dense_proj_plan": [_i32, _i32, _i32, _i32, _p, _p, _p, _p],
    "dense_proj_tune": [_i32, _i32],
    "spike_quantize_int8": [_p, _i32, _i32, _i32, _p, _p, _p],
    "spike_check_scale_shape": [_i32, _i32, _i32, _i32, _i32],
    "head_verify_forward": [_p, _p, _i32, _i32, _p, _i32, ctypes.c_float, _p, _p, _p, _p, _p, _p],
    "head_verify_workspace_bytes": [],
}
for _name, _args in _sig.items():
    getattr(_lib, _name).argtypes = _args
    getattr(_lib, _name).restype = ctypes.c_int
_lib.spike_proj_last_error.argtypes = []
_lib.spike_proj_last_error.restype = ctypes.c_char_p
_lib.head_verify_workspace_bytes.restype = ctypes.c_int64


class SpikeError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where} failed with code {code}: {spike_proj_last_error()}")


def _check(rc: int, where: str) -> None:
    if rc != SPIKE_OK:
        raise SpikeError(rc, where)


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _dev_ptr(t: torch.Tensor, name: str, nbytes: int | None = None) -> int:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if nbytes is not None and t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes, needs {nbytes}")
    return t.data_ptr()


def words_per_row(K: int) -> int:
    return (int(K) + 63) // 64


class SpikeProj:
    """Handle returned by spike_proj_create.  Holds the borrowed W and scale
    tensors so they outlive the handle."""

    def __init__(self, ptr: int, W: torch.Tensor, scale: torch.Tensor):
        self.ptr, self.W, self.scale = ptr, W, scale
        self.K, self.N = W.shape
        self.max_B = SPIKE_DEFAULT_MAX_B

    def close(self):
        if self.ptr:
            _check(_lib.spike_proj_destroy(self.ptr), "spike_proj_destroy")
            self.ptr = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _check_operands(W: torch.Tensor, scale: torch.Tensor) -> None:
    if W.dtype != torch.int8 or W.dim() != 2:
        raise TypeError("W must be an int8 tensor [K, N]")
    if scale.dtype != torch.float32 or scale.shape != (W.shape[1],):
        raise TypeError(f"scale must be float32 [N={W.shape[1]}]")


def spike_proj_create(W: torch.Tensor, scale: torch.Tensor) -> SpikeProj:
    """W: int8 [K, N] (column-major storage of the [N, K] weight), scale: float32 [N]."""
    _check_operands(W, scale)
    out = _p()
    _check(_lib.spike_proj_create(_dev_ptr(W, "W"), _dev_ptr(scale, "scale"), W.shape[0], W.shape[1],
                                  ctypes.byref(out)), "spike_proj_create")
    return SpikeProj(out.value, W, scale)


SPIKE_CREATE_GATHER_ONLY = 1


def spike_proj_create_reserved(W: torch.Tensor, scale: torch.Tensor, max_B: int, gather_only: bool = False) -> SpikeProj:
    """spike_proj_create with a workspace for max_B rows; gather_only: never hold the matrix-core copy."""
    _check_operands(W, scale)
    out = _p()
    _check(_lib.spike_proj_create_reserved(_dev_ptr(W, "W"), _dev_ptr(scale, "scale"), W.shape[0], W.shape[1],
                                           int(max_B), SPIKE_CREATE_GATHER_ONLY if gather_only else 0,
                                           ctypes.byref(out)), "spike_proj_create_reserved")
    h = SpikeProj(out.value, W, scale)
    h.max_B = int(max_B)
    return h


def spike_proj_reserve(h: SpikeProj, max_B: int) -> None:
    _check(_lib.spike_proj_reserve(h.ptr, int(max_B)), "spike_proj_reserve")
    h.max_B = int(max_B)


def spike_proj_forward(h: SpikeProj, mask: torch.Tensor, B: int, out: torch.Tensor, stream=None) -> None:
    """mask: B rows of ceil(K/64) 64-bit words (any integer dtype, same bytes); out: float32 [B, N]."""
    if out.dtype != torch.float32:
        raise TypeError("out must be float32")
    _check(_lib.spike_proj_forward(h.ptr, _dev_ptr(mask, "mask", B * words_per_row(h.K) * 8), int(B),
                                   _dev_ptr(out, "out", B * h.N * 4), _stream(stream)), "spike_proj_forward")


def spike_proj_forward_acc(h: SpikeProj, mask: torch.Tensor, B: int, acc: torch.Tensor, stream=None) -> None:
    if acc.dtype != torch.int32:
        raise TypeError("acc must be int32")
    _check(_lib.spike_proj_forward_acc(h.ptr, _dev_ptr(mask, "mask", B * words_per_row(h.K) * 8), int(B),
                                       _dev_ptr(acc, "acc", B * h.N * 4), _stream(stream)), "spike_proj_forward_acc")


SPIKE_STATIC_SCRATCH_WORDS = 1 << 20


def spike_proj_forward_noalloc(W: torch.Tensor, scale: torch.Tensor, mask: torch.Tensor, B: int, out: torch.Tensor,
                               stream=None) -> None:
    """Handle-free forward on the library's static scratch (no device allocation)."""
    _check_operands(W, scale)
    K, N = W.shape
    if out.dtype != torch.float32:
        raise TypeError("out must be float32")
    _check(_lib.spike_proj_forward_noalloc(_dev_ptr(W, "W"), _dev_ptr(scale, "scale"), int(K), int(N),
                                           _dev_ptr(mask, "mask", B * words_per_row(K) * 8), int(B),
                                           _dev_ptr(out, "out", B * N * 4), _stream(stream)),
           "spike_proj_forward_noalloc")


def spike_proj_destroy(h: SpikeProj) -> None:
    h.close()


def spike_proj_tune(h: SpikeProj, key: int, value: int) -> None:
    _check(_lib.spike_proj_tune(h.ptr, int(key), int(value)), "spike_proj_tune")


def spike_compact(mask: torch.Tensor, B: int, K: int, active_idx: torch.Tensor, active_count: torch.Tensor,
                  stream=None) -> None:
    if active_idx.dtype != torch.int32 or active_count.dtype != torch.int32:
        raise TypeError("active_idx and active_count must be int32")
    _check(_lib.spike_compact(_dev_ptr(mask, "mask", B * words_per_row(K) * 8), int(B), int(K),
                              _dev_ptr(active_idx, "active_idx", B * K * 4),
                              _dev_ptr(active_count, "active_count", B * 4), _stream(stream)), "spike_compact")


def _handle_array(handles):
    arr = (_p * len(handles))(*[h.ptr for h in handles])
    return arr


def spike_stack_forward(handles, masks: torch.Tensor, B: int, out: torch.Tensor, stream=None) -> None:
    """Run the projections in order; masks/out packed per projection (see the header)."""
    arr = _handle_array(handles)
    mwords = sum(B * words_per_row(h.K) for h in handles)
    ofl = sum(B * h.N for h in handles)
    _check(_lib.spike_stack_forward(arr, len(handles), _dev_ptr(masks, "masks", mwords * 8), int(B),
                                    _dev_ptr(out, "out", ofl * 4), _stream(stream)), "spike_stack_forward")


def spike_stack_forward_fused(handles, masks: torch.Tensor, B: int, out: torch.Tensor, stream=None) -> None:
    """All projections in one matrix-core launch (inputs all given); same layout as spike_stack_forward."""
    arr = _handle_array(handles)
    mwords = sum(B * words_per_row(h.K) for h in handles)
    ofl = sum(B * h.N for h in handles)
    _check(_lib.spike_stack_forward_fused(arr, len(handles), _dev_ptr(masks, "masks", mwords * 8), int(B),
                                          _dev_ptr(out, "out", ofl * 4), _stream(stream)), "spike_stack_forward_fused")


class SpikeStream:
    def __init__(self, ptr: int, handles, n_proj: int, n_sets: int, n_tokens: int):
        self.ptr, self.handles = ptr, list(handles)
        self.n_proj, self.n_sets, self.n_tokens = n_proj, n_sets, n_tokens
        self.token_words = sum(words_per_row(h.K) for h in self.handles[:n_proj])
        self.token_out = sum(h.N for h in self.handles[:n_proj])

    def close(self):
        if self.ptr:
            _check(_lib.spike_stream_destroy(self.ptr), "spike_stream_destroy")
            self.ptr = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def spike_stream_create(handles, n_proj: int, n_sets: int, n_tokens: int) -> SpikeStream:
    if len(handles) != n_proj * n_sets:
        raise ValueError("need n_proj * n_sets handles")
    out = _p()
    _check(_lib.spike_stream_create(_handle_array(handles), int(n_proj), int(n_sets), int(n_tokens),
                                    ctypes.byref(out)), "spike_stream_create")
    return SpikeStream(out.value, handles, n_proj, n_sets, n_tokens)


def spike_stream_forward(s: SpikeStream, masks: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    _check(_lib.spike_stream_forward(s.ptr, _dev_ptr(masks, "masks", s.n_tokens * s.token_words * 8),
                                     _dev_ptr(out, "out", s.n_tokens * s.token_out * 4), _stream(stream)),
           "spike_stream_forward")


def spike_stream_tune(s: SpikeStream, key: int, value: int) -> None:
    _check(_lib.spike_stream_tune(s.ptr, int(key), int(value)), "spike_stream_tune")


def spike_stream_destroy(s: SpikeStream) -> None:
    s.close()


def spike_proj_last_error() -> str:
    return _lib.spike_proj_last_error().decode()


def spike_proj_shapes() -> list:
    """Launch-shape codes instantiated by the library."""
    n = _lib.spike_proj_shapes(None, 0)
    buf = (ctypes.c_int32 * n)()
    _lib.spike_proj_shapes(buf, n)
    return list(buf)


def spike_mfma_plans() -> list:
    """Matrix-core plans instantiated by the library, as dicts."""
    n = _lib.spike_mfma_plans(None, 0)
    buf = (ctypes.c_int32 * n)()
    _lib.spike_mfma_plans(buf, n)
    return [decode_plan(c) for c in buf]


def decode_plan(code: int) -> dict:
    return {"rt": code & 15, "cs": (code >> 4) & 15, "kw": (code >> 8) & 255, "d": (code >> 16) & 255,
            "preload": bool((code >> 24) & 1), "direct": bool((code >> 25) & 1)}


def spike_proj_plan_query(K: int, N: int, B: int):
    """(path, plan dict or None) that AUTO takes for B rows of a K x N projection."""
    path, plan = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.spike_proj_plan_query(int(K), int(N), int(B), ctypes.byref(path), ctypes.byref(plan)),
           "spike_proj_plan_query")
    return path.value, (decode_plan(plan.value) if plan.value else None)


def dense_proj_forward(Q: torch.Tensor, scale: torch.Tensor, x: torch.Tensor, B: int, y: torch.Tensor,
                       stream=None) -> None:
    """y[:B] = scale * (x[:B] @ float(Q).T) for row-major INT8 Q [M][K] (dense_proj.h)."""
    if Q.dtype != torch.int8 or Q.dim() != 2:
        raise TypeError("Q must be a 2-D int8 tensor [M][K]")
    M, K = Q.shape
    if scale.dtype != torch.float32 or scale.numel() != M:
        raise TypeError("scale must be float32 with M entries")
    if x.dtype != torch.float32 or y.dtype != torch.float32:
        raise TypeError("x and y must be float32")
    B = int(B)
    _check(_lib.dense_proj_forward(_dev_ptr(Q, "Q"), _dev_ptr(scale, "scale"), int(K), int(M),
                                   _dev_ptr(x, "x", B * K * 4), B, _dev_ptr(y, "y", B * M * 4), _stream(stream)),
           "dense_proj_forward")


def dense_proj_plan(K: int, M: int, B: int, q_align: int = 16) -> dict:
    """Launch shape of the first launch dense_proj_forward makes (host-only)."""
    out = [ctypes.c_int32() for _ in range(4)]
    _check(_lib.dense_proj_plan(int(K), int(M), int(B), int(q_align), *[ctypes.byref(o) for o in out]),
           "dense_proj_plan")
    return dict(zip(("kernel", "vec", "rows_per_launch", "workgroups"), (o.value for o in out)))


def dense_proj_tune(key: int, value: int) -> None:
    _check(_lib.dense_proj_tune(int(key), int(value)), "dense_proj_tune")


def spike_quantize_int8(W: torch.Tensor, layout: int, Q: torch.Tensor, scale: torch.Tensor, stream=None) -> None:
    """Symmetric per-channel INT8 quantization of W [M][K] (quantize.h): Q
    int8 row-major [M][K] or column-major [K][M], scale float32 [M]."""
    if W.dtype != torch.float32 or W.dim() != 2:
        raise TypeError("W must be a 2-D float32 tensor [M][K]")
    M, K = W.shape
    if Q.dtype != torch.int8 or scale.dtype != torch.float32:
        raise TypeError("Q must be int8 and scale float32")
    _check(_lib.spike_quantize_int8(_dev_ptr(W, "W"), int(M), int(K), int(layout), _dev_ptr(Q, "Q", M * K),
                                    _dev_ptr(scale, "scale", M * 4), _stream(stream)), "spike_quantize_int8")


def spike_check_scale_shape(M: int, K: int, group: int, scale_rows: int, scale_cols: int) -> None:
    _check(_lib.spike_check_scale_shape(int(M), int(K), int(group), int(scale_rows), int(scale_cols)),
           "spike_check_scale_shape")


def head_verify_workspace(device=None) -> torch.Tensor:
    """A workspace for head_verify_forward on `device` (head_verify.h)."""
    n = int(_lib.head_verify_workspace_bytes())
    return torch.empty(n, dtype=torch.uint8, device=device if device is not None else "cuda")


_head_workspaces: dict = {}


def head_verify_forward(Q: torch.Tensor, scale: torch.Tensor, x: torch.Tensor, top_k: int, threshold: float,
                        logits: torch.Tensor, cand: torch.Tensor, cand_logits: torch.Tensor, result: torch.Tensor,
                        stream=None, workspace: torch.Tensor | None = None) -> None:
    """INT8-activation head, top-k candidates, gap gate, FP32 recompute
    (head_verify.h).  Without `workspace`, one kept per device is used (calls
    on several streams of one device then need their own)."""
    if Q.dtype != torch.int8 or Q.dim() != 2:
        raise TypeError("Q must be a 2-D int8 tensor [V][K]")
    V, K = Q.shape
    for t, name, dt in ((scale, "scale", torch.float32), (x, "x", torch.float32), (logits, "logits", torch.float32),
                        (cand, "cand", torch.int32), (cand_logits, "cand_logits", torch.float32),
                        (result, "result", torch.int32)):
        if t.dtype != dt:
            raise TypeError(f"{name} must be {dt}")
    k = int(top_k)
    if workspace is None:
        dev = Q.device.index if Q.device.index is not None else torch.cuda.current_device()
        workspace = _head_workspaces.get(dev)
        if workspace is None:
            workspace = _head_workspaces[dev] = head_verify_workspace(torch.device("cuda", dev))
    n_ws = int(_lib.head_verify_workspace_bytes())
    _check(_lib.head_verify_forward(_dev_ptr(Q, "Q"), _dev_ptr(scale, "scale", V * 4), int(K), int(V),
                                    _dev_ptr(x, "x", K * 4), k, float(threshold), _dev_ptr(logits, "logits", V * 4),
                                    _dev_ptr(cand, "cand", k * 4), _dev_ptr(cand_logits, "cand_logits", k * 4),
                                    _dev_ptr(result, "result", 8), _dev_ptr(workspace, "workspace", n_ws),
                                    _stream(stream)), "head_verify_forward")


def spike_proj_abi_version() -> int:
    return _lib.spike_proj_abi_version()


def raw_library():
    """The loaded ctypes library (for ABI tests that call entry points directly)."""
    return _lib
