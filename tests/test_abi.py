"""The C-ABI library: it loads, exports every entry point the header
declares, and rejects bad arguments before touching the GPU (no GPU needed:
every call here returns from argument validation)."""
import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def sp():
    from paper_2606_03026_amd import _binding
    return _binding


def declared_functions():
    names = set()
    for hdr in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = re.sub(r"/\*.*?\*/", "", open(hdr).read(), flags=re.S)
        names |= set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*((?:spike|dense|head)_\w+)\s*\(", text, flags=re.M))
    return sorted(names)


def test_header_declares_the_entry_points():
    names = declared_functions()
    for required in ("spike_proj_create", "spike_proj_forward", "spike_proj_destroy", "dense_proj_forward"):
        assert required in names


def test_library_exports_every_declared_symbol(sp):
    lib = sp.raw_library()
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, f"not exported: {missing}"
    assert set(sp.EXPORTED) == set(declared_functions())


def test_abi_version(sp):
    assert sp.spike_proj_abi_version() == 2


def test_argument_validation_before_any_hip_call(sp):
    lib = sp.raw_library()
    out = ctypes.c_void_p()
    dummy = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    assert lib.spike_proj_create(None, dummy, 4, 4, ctypes.byref(out)) == sp.SPIKE_EINVAL
    assert out.value is None
    assert "null" in sp.spike_proj_last_error()
    assert lib.spike_proj_create(dummy, dummy, 0, 4, ctypes.byref(out)) == sp.SPIKE_EINVAL
    assert lib.spike_proj_create(dummy, dummy, 4, 0, ctypes.byref(out)) == sp.SPIKE_EINVAL
    assert lib.spike_proj_create(dummy, dummy, (1 << 24) + 1, 4, ctypes.byref(out)) == sp.SPIKE_EINVAL
    assert "K" in sp.spike_proj_last_error()
    assert lib.spike_proj_create(dummy, dummy, 4, 4, None) == sp.SPIKE_EINVAL
    assert lib.spike_proj_forward(None, dummy, 1, dummy, None) == sp.SPIKE_EINVAL
    assert lib.spike_proj_forward_acc(None, dummy, 1, dummy, None) == sp.SPIKE_EINVAL
    assert lib.spike_proj_reserve(None, 8) == sp.SPIKE_EINVAL
    assert lib.spike_proj_tune(None, sp.SPIKE_TUNE_PATH, 0) == sp.SPIKE_EINVAL
    assert lib.spike_proj_destroy(None) == sp.SPIKE_OK
    assert lib.spike_compact(dummy, -1, 64, dummy, dummy, None) == sp.SPIKE_EINVAL
    assert lib.spike_compact(dummy, 1, 0, dummy, dummy, None) == sp.SPIKE_EINVAL
    assert lib.spike_compact(dummy, 0, 64, None, None, None) == sp.SPIKE_OK  # B = 0 is a no-op
    assert lib.spike_stack_forward(None, 2, dummy, 1, dummy, None) == sp.SPIKE_EINVAL
    assert lib.spike_stream_create(None, 2, 1, 1, ctypes.byref(out)) == sp.SPIKE_EINVAL
    assert lib.spike_stream_forward(None, dummy, dummy, None) == sp.SPIKE_EINVAL
    assert lib.spike_stream_destroy(None) == sp.SPIKE_OK


def test_product_path_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2606_03026_amd")
    for path in glob.glob(os.path.join(pkg, "**", "*"), recursive=True):
        if os.path.isfile(path) and path.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
            text = open(path).read()
            assert not re.search(r"^\s*(import|from)\s+oracle", text, flags=re.M), path
            assert "spike_oracle" not in text, path
    hdr = open(os.path.join(ROOT, "include", "spike_proj.h")).read()
    assert "oracle" not in hdr


def test_automatic_matrix_core_plans_are_instantiated(sp):
    """For every shape and batch the host-side planner sends to the matrix
    cores, the plan is one the library instantiates; the decode shapes and
    the prefill shape go where the design puts them (no GPU needed)."""
    plans = {tuple(p.values()) for p in sp.spike_mfma_plans()}
    for K in (1, 63, 64, 65, 100, 300, 1000, 1536, 2048, 4097, 6144, 16384, 20000, 40000):
        for N in (16, 64, 100, 192, 1536, 6144, 1 << 20):
            for B in (1, 4, 5, 16, 17, 64, 65, 130, 512, 4096):
                path, plan = sp.spike_proj_plan_query(K, N, B)
                if path == sp.SPIKE_PATH_MFMA:
                    assert tuple(plan.values()) in plans, (K, N, B, plan)
                    assert N % 16 == 0
                else:
                    assert path == sp.SPIKE_PATH_GATHER
                    # the gather serves what the matrix cores cannot: N not a
                    # multiple of 16, a packed copy of 2^31 bytes or more, or
                    # rows whose staged spike words (16 rows of ceil(K/64) | 1
                    # words) do not fit the 64 KB LDS budget
                    staged = 16 * (((K + 63) // 64) | 1) * 8
                    assert N % 16 != 0 or (K + 63) // 64 * 64 * N >= 1 << 31 or staged > 60000, (K, N, B)
    # batch-1 decode calls and small batches: one channel set per workgroup
    for K in (1536, 6144):
        for B in (1, 4, 16):
            path, plan = sp.spike_proj_plan_query(K, 1536, B)
            assert path == sp.SPIKE_PATH_MFMA and plan["rt"] == 1 and plan["cs"] == 1
        path, plan = sp.spike_proj_plan_query(K, 1536, 64)
        assert path == sp.SPIKE_PATH_MFMA and plan["rt"] == 1
    path, plan = sp.spike_proj_plan_query(6144, 1536, 512)
    assert path == sp.SPIKE_PATH_MFMA and plan["rt"] == 4
    assert sp.spike_proj_plan_query(1536, 1000, 1)[0] == sp.SPIKE_PATH_GATHER


def test_dense_argument_validation_before_any_hip_call(sp):
    lib = sp.raw_library()
    d = 0x1000  # never dereferenced: validation fails first
    assert lib.dense_proj_forward(d, d, 0, 4, d, 1, d, None) == sp.SPIKE_EINVAL
    assert "K = 0" in sp.spike_proj_last_error()
    assert lib.dense_proj_forward(d, d, sp.DENSE_MAX_K + 1, 4, d, 1, d, None) == sp.SPIKE_EINVAL
    assert lib.dense_proj_forward(d, d, 64, 0, d, 1, d, None) == sp.SPIKE_EINVAL
    assert lib.dense_proj_forward(d, d, 16000, 1 << 18, d, 1, d, None) == sp.SPIKE_EUNSUPPORTED
    assert "exceeds" in sp.spike_proj_last_error()
    assert lib.dense_proj_forward(d, d, 64, 4, d, -1, d, None) == sp.SPIKE_EINVAL
    assert lib.dense_proj_forward(d, d, 64, 4, d, sp.DENSE_MAX_B + 1, d, None) == sp.SPIKE_EINVAL
    assert lib.dense_proj_forward(None, d, 64, 4, d, 1, d, None) == sp.SPIKE_EINVAL
    assert "null" in sp.spike_proj_last_error()
    assert lib.dense_proj_forward(d, d, 64, 4, d + 2, 1, d, None) == sp.SPIKE_EINVAL
    assert lib.dense_proj_forward(None, None, 64, 4, None, 0, None, None) == sp.SPIKE_OK  # B = 0: nothing to do
    assert sp.spike_proj_last_error() == ""


def test_dense_plans(sp):
    """Kernel and load width follow K and Q's alignment only; a launch takes up
    to 4 (register kernel) or 8 (staged kernel) batch rows; the vocabulary head
    spreads over at least two workgroups per CU."""
    reg, staged = sp.DENSE_KERNEL_REGISTER, sp.DENSE_KERNEL_STAGED
    head = sp.dense_proj_plan(1536, 57344, 1)
    assert (head["kernel"], head["vec"]) == (reg, 16)
    assert head["workgroups"] >= 512
    for B in (1, 2, 3, 8, 13):
        assert sp.dense_proj_plan(1536, 57344, B)["kernel"] == reg
    assert sp.dense_proj_plan(1536, 57344, 1, q_align=4)["kernel"] == staged
    assert sp.dense_proj_plan(1536, 57344, 1, q_align=4)["vec"] == 4
    assert sp.dense_proj_plan(1536, 57344, 1, q_align=8)["vec"] == 4
    assert sp.dense_proj_plan(1540, 100, 1)["vec"] == 4
    assert sp.dense_proj_plan(1537, 100, 1)["vec"] == 1
    assert sp.dense_proj_plan(1536, 100, 1, q_align=2)["vec"] == 1
    assert sp.dense_proj_plan(4096, 100, 1)["kernel"] == reg
    assert sp.dense_proj_plan(4112, 100, 1)["kernel"] == staged
    assert [sp.dense_proj_plan(512, 100, B)["rows_per_launch"] for B in (1, 2, 3, 5, 8)] == [1, 2, 4, 4, 4]
    assert [sp.dense_proj_plan(1536, 100, B)["rows_per_launch"] for B in (1, 2, 3)] == [1, 2, 2]
    assert [sp.dense_proj_plan(2048, 100, B)["rows_per_launch"] for B in (1, 2, 3)] == [1, 1, 1]
    assert [sp.dense_proj_plan(1540, 100, B)["rows_per_launch"] for B in (1, 2, 3, 5, 8, 13)] == [1, 2, 4, 8, 8, 8]
    assert sp.dense_proj_plan(sp.DENSE_MAX_K, 3, 8)["rows_per_launch"] == 1  # LDS holds one row of the largest K
    with pytest.raises(sp.SpikeError):
        sp.dense_proj_plan(64, 4, 1, q_align=3)
    try:
        sp.dense_proj_tune(sp.DENSE_TUNE_KERNEL, staged)
        assert sp.dense_proj_plan(1536, 57344, 1)["kernel"] == staged
        sp.dense_proj_tune(sp.DENSE_TUNE_WG_PER_CU, 2)
        sp.dense_proj_tune(sp.DENSE_TUNE_KERNEL, 0)
        assert sp.dense_proj_plan(1536, 57344, 1)["workgroups"] == 512
        with pytest.raises(sp.SpikeError):
            sp.dense_proj_tune(sp.DENSE_TUNE_KERNEL, 7)
        with pytest.raises(sp.SpikeError):
            sp.dense_proj_tune(99, 0)
    finally:
        sp.dense_proj_tune(sp.DENSE_TUNE_KERNEL, 0)
        sp.dense_proj_tune(sp.DENSE_TUNE_WG_PER_CU, 0)


def test_create_rejects_unknown_flags(sp):
    lib = sp.raw_library()
    out = ctypes.c_void_p()
    dummy = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    assert lib.spike_proj_create_reserved(dummy, dummy, 4, 4, 1, 2, ctypes.byref(out)) == sp.SPIKE_EINVAL
    assert "flags" in sp.spike_proj_last_error()
    assert lib.spike_proj_create_reserved(dummy, dummy, 4, 4, 0, 0, ctypes.byref(out)) == sp.SPIKE_EINVAL


def test_quantizer_argument_validation_before_any_hip_call(sp):
    lib = sp.raw_library()
    d = 0x1000  # never dereferenced: validation fails first
    assert lib.spike_quantize_int8(d, 0, 4, 0, d, d, None) == sp.SPIKE_EINVAL
    assert lib.spike_quantize_int8(d, 4, 0, 0, d, d, None) == sp.SPIKE_EINVAL
    assert lib.spike_quantize_int8(d, 1 << 16, 1 << 16, 0, d, d, None) == sp.SPIKE_EINVAL
    assert "2^31" in sp.spike_proj_last_error()
    assert lib.spike_quantize_int8(d, 4, 4, 2, d, d, None) == sp.SPIKE_EINVAL
    assert "layout" in sp.spike_proj_last_error()
    assert lib.spike_quantize_int8(None, 4, 4, 0, d, d, None) == sp.SPIKE_EINVAL
    assert lib.spike_quantize_int8(d + 2, 4, 4, 0, d, d, None) == sp.SPIKE_EINVAL


def test_scale_shape_check_names_the_transposed_export(sp):
    """The paper's withdrawn export: an FFN down weight [1536][6144] with
    group 32 needs scales [1536][192]; scales taken after transposing have
    shape [6144][48] -- the same element count -- and must be refused."""
    sp.spike_check_scale_shape(1536, 6144, 32, 1536, 192)
    sp.spike_check_scale_shape(1536, 6144, 6144, 1536, 1)  # per-channel
    with pytest.raises(sp.SpikeError, match="transposed"):
        sp.spike_check_scale_shape(1536, 6144, 32, 6144, 48)
    with pytest.raises(sp.SpikeError, match="transposed"):
        sp.spike_check_scale_shape(1536, 6144, 6144, 6144, 1)
    with pytest.raises(sp.SpikeError, match="does not match"):
        sp.spike_check_scale_shape(1536, 6144, 32, 1536, 193)
    with pytest.raises(sp.SpikeError):
        sp.spike_check_scale_shape(1536, 6144, 0, 1536, 192)
    sp.spike_check_scale_shape(1536, 1536, 32, 1536, 48)  # square: the shapes coincide


def test_head_verify_argument_validation_before_any_hip_call(sp):
    lib = sp.raw_library()
    d = 0x1000  # never dereferenced: validation fails first
    f = lib.head_verify_forward
    assert f(d, d, 24, 100, d, 8, 0.5, d, d, d, d, d, None) == sp.SPIKE_EINVAL  # K % 16
    assert f(d, d, 4112, 100, d, 8, 0.5, d, d, d, d, d, None) == sp.SPIKE_EINVAL  # K too large
    assert f(d, d, 1536, 0, d, 8, 0.5, d, d, d, d, d, None) == sp.SPIKE_EINVAL
    assert f(d, d, 1536, 100, d, 0, 0.5, d, d, d, d, d, None) == sp.SPIKE_EINVAL
    assert f(d, d, 1536, 100, d, 65, 0.5, d, d, d, d, d, None) == sp.SPIKE_EINVAL
    assert f(d, d, 1536, 5, d, 6, 0.5, d, d, d, d, d, None) == sp.SPIKE_EINVAL  # top_k > V
    assert f(d, d, 1536, 100, d, 8, float("nan"), d, d, d, d, d, None) == sp.SPIKE_EINVAL
    assert "NaN" in sp.spike_proj_last_error()
    assert f(d + 4, d, 1536, 100, d, 8, 0.5, d, d, d, d, d, None) == sp.SPIKE_EINVAL
    assert "16-byte" in sp.spike_proj_last_error()
    assert f(d, d, 1536, 100, d, 8, 0.5, None, d, d, d, d, None) == sp.SPIKE_EINVAL
    assert f(d, d, 1536, 100, d, 8, 0.5, d, d, d, d, None, None) == sp.SPIKE_EINVAL  # no workspace
    assert f(d, d, 1536, 100, d, 8, 0.5, d, d, d, d, d + 8, None) == sp.SPIKE_EINVAL
    assert "workspace" in sp.spike_proj_last_error()
    n = lib.head_verify_workspace_bytes()
    assert 0 < n < 1 << 20 and n % 16 == 0
