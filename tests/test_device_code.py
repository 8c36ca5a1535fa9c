"""The gfx950 code built here holds no packed FP32 instruction.

Packed FP32 arithmetic (and the packed 32-bit move of the same instruction group) is disabled
for all device code, yet the compiler still emits the packed move for some vector shuffles, so
the build disassembles every code object it makes and rejects one that holds such an
instruction. These tests check that the built executor passes and that a kernel which does
hold one is rejected (it is only compiled, never run).
"""
import os
import subprocess

import pytest

from paper_2608_00358_amd import _build

SHUFFLE = r"""
#include <hip/hip_runtime.h>
#include <stdint.h>
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__global__ void shuffle(const u32x4* a, u32x4* b, uint32_t s, uint32_t n) {
    for (uint32_t i = threadIdx.x; i < n; i += blockDim.x) {
        const u32x4 A = a[i], B = a[i + 1];
        b[i] = s == 1 ? u32x4{A[1], A[2], A[3], B[0]}
             : s == 2 ? u32x4{A[2], A[3], B[0], B[1]} : u32x4{A[3], B[0], B[1], B[2]};
    }
}
"""


def _hipcc():
    try:
        return _build._hipcc()
    except RuntimeError:
        pytest.skip("hipcc is not available")


def test_built_executor_holds_no_packed_fp32():
    obj = os.path.join(_build.OBJDIR, "executor.hip.o")
    if not os.path.exists(obj):
        pytest.skip("the executor is not built")
    _build.check_device_code(obj)


def test_check_rejects_a_kernel_with_a_packed_move(tmp_path):
    src, obj = tmp_path / "shuffle.hip", tmp_path / "shuffle.o"
    src.write_text(SHUFFLE)
    res = subprocess.run([_hipcc(), *_build.HIPCC_FLAGS, "-x", "hip", "-c", str(src), "-o", str(obj)],
                         capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    with pytest.raises(RuntimeError, match="v_pk_mov_b32"):
        _build.check_device_code(str(obj))
