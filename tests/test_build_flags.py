"""The device code is built without packed FP32 instructions (v_pk_add_f32,
v_pk_mul_f32, v_pk_fma_f32): the library's hipcc flags disable the target
feature that lets the compiler form them.  Checked on the gfx950 assembly of
every library source (no GPU needed), with a control kernel showing that the
same compiler does form them when the flag is absent."""
import os
import re
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2606_03026_amd import build

PACKED = re.compile(r"\bv_pk_(add|mul|fma)_f32\b")
CONTROL = r"""
#include <hip/hip_runtime.h>
__global__ void k(const float2* a, const float2* b, float2* c)
{
    const int i = threadIdx.x;
    const float2 x = a[i], y = b[i];
    c[i] = make_float2(x.x * y.x + 1.0f, x.y * y.y + 1.0f);
}
"""

pytestmark = pytest.mark.skipif(not os.path.exists(build.HIPCC) and shutil.which("hipcc") is None,
                                reason="hipcc not installed")


def device_asm(src: str, flags, tmp_path, tag: str) -> str:
    out = tmp_path / f"{tag}.s"
    cmd = [build.HIPCC, *[f for f in flags if f not in ("-shared", "-fPIC")], "--cuda-device-only", "-S",
           "-o", str(out), src]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-2000:]
    return out.read_text()


def test_control_kernel_gets_packed_fp32_without_the_flag(tmp_path):
    src = tmp_path / "control.hip"
    src.write_text(CONTROL)
    base = [f for f in build.FLAGS if f not in ("-Xclang", "-target-feature", "-packed-fp32-ops")]
    assert PACKED.search(device_asm(str(src), base, tmp_path, "without"))
    assert not PACKED.search(device_asm(str(src), build.FLAGS, tmp_path, "with"))


def test_library_device_code_has_no_packed_fp32(tmp_path):
    with ThreadPoolExecutor(max_workers=min(4, len(build.SOURCES))) as ex:
        asms = list(ex.map(lambda s: (s, device_asm(s, build.FLAGS, tmp_path, os.path.basename(s))), build.SOURCES))
    for src, asm in asms:
        assert ".amdhsa_kernel" in asm, f"no kernels found in {src}"
        hits = PACKED.findall(asm)
        assert not hits, f"{os.path.basename(src)}: packed FP32 instructions {hits[:5]}"
