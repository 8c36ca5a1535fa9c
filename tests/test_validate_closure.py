"""The validator's two forms of the dependency closure (bit matrices up to 24 000 steps, a
per-pair backward search beyond) give the same verdicts, and programs past the bit matrices'
limit validate.

The native driver compiles collectives with the library's lowering, fusion and finalisation and
validates each program, and mutants of it that lack an ordering, both ways.
"""
import os
import shutil
import subprocess

import pytest

import paper_2608_00358_amd as H
from test_compiler import fake_bufs

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "..", "paper_2608_00358_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_bit_matrices_and_search_agree(tmp_path):
    exe = str(tmp_path / "validate_closure")
    subprocess.run(["g++", "-std=c++17", "-O2", "-I", CSRC, os.path.join(HERE, "native", "validate_closure.cpp"),
                    os.path.join(CSRC, "compiler.cpp"), os.path.join(CSRC, "validate.cpp"), "-o", exe], check=True)
    out = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    print(out.stdout[-2000:])
    assert out.returncode == 0, out.stdout[-2000:]
    assert "mismatched 0" in out.stdout


@pytest.mark.parametrize("phases", ["one", "auto"])
def test_program_past_the_bit_matrices_validates(phases):
    # ring all-reduce of 32 ranks, 49 153 fp32 in 512-byte chunks, unfused: 24 800 steps
    # (31 reduce steps and 31 forwarding copies of 400 chunks), every wait inside one launch
    P = 32
    with H.Comm(P, device=H.NO_DEVICE, algo="ring", fuse=0, chunk_bytes=512, validate=1, phases=phases) as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), 49153, "fp32")
        info = c.last_program()
    assert info["num_descs"] == 24800 and info["num_phases"] == 1 and info["num_deps"] > 0
