"""The built library's GPU code (CPU only: disassembles code built here).

Every HIP source is compiled without packed FP32 instructions
(v_pk_add_f32, v_pk_mul_f32, v_pk_fma_f32): the build passes the target
feature off, and this checks that the gfx950 code objects inside libeqb.so
really contain none of them."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_28053_amd", "libeqb.so")
OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"


def test_no_packed_fp32_instructions_in_device_code(tmp_path):
    if not os.path.exists(OBJDUMP):
        pytest.skip("llvm-objdump not installed")
    assert os.path.exists(LIB), "libeqb.so is not built"
    lib = tmp_path / "libeqb.so"
    shutil.copy(LIB, lib)
    subprocess.run([OBJDUMP, "--offloading", str(lib)], check=True, capture_output=True, cwd=tmp_path)
    objs = sorted(glob.glob(str(tmp_path / "libeqb.so.*gfx950")))
    assert objs, "no gfx950 code object in the library"
    total = 0
    for co in objs:
        asm = subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", co], check=True, capture_output=True,
                             text=True).stdout
        total += asm.count("v_med3_f32")
        for op in ("v_pk_add_f32", "v_pk_mul_f32", "v_pk_fma_f32"):
            assert op not in asm, f"{op} in {os.path.basename(co)}"
    assert total > 1000          # the routing kernels were disassembled
