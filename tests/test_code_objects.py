"""The gfx950 code objects this repository builds (CPU; the library's own
objects in paper_2609_35115_amd/_build, release and checked builds): each is
taken from its object's .hip_fatbin section, disassembled with the ROCm LLVM
tools, and must contain
  * no scalar-memory write of any kind (scalar stores and atomics, scalar
    buffer and scratch stores, scalar cache write-back or discard): the
    kernels write through vector memory only;
  * no packed fp32 VALU operation (the build turns the packed-fp32-ops
    target feature off; the compiler must not have produced one anyway);
and the MFMA kernels must be there (the checks ran on real code)."""
from __future__ import annotations

import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OBJDIR = os.path.join(ROOT, "paper_2609_35115_amd", "_build")
LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"
OBJECTS = ["libdc_so_dc_kernels.o", "libdc_so_flow_kernels.o", "libdc_debug_dc_kernels.o",
           "libdc_so_dc_runtime.o", "libdc_so_flow_runtime.o"]

SCALAR_WRITE = re.compile(r"\bs_(store|atomic|dcache_wb|dcache_discard|buffer_store|buffer_atomic|scratch_store)\w*")
PACKED_F32 = re.compile(r"\bv_pk_(add|mul|fma)_f32\b")


def _disassemble(obj: str, tmp) -> str | None:
    fat = str(tmp / (os.path.basename(obj) + ".fatbin"))
    r = subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fat}", obj, str(tmp / "x.o")],
                       capture_output=True, text=True)
    if r.returncode != 0:
        return None   # no device code in this object
    co = str(tmp / (os.path.basename(obj) + ".co"))
    subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o", f"--input={fat}",
                    f"--targets={TARGET}", f"--output={co}"], check=True, capture_output=True)
    r = subprocess.run([f"{LLVM}/llvm-objdump", "-d", "--mcpu=gfx950", co], check=True, capture_output=True,
                       text=True)
    return r.stdout


@pytest.mark.parametrize("name", OBJECTS)
def test_code_object_has_no_scalar_writes_or_packed_fp32(name, tmp_path):
    obj = os.path.join(OBJDIR, name)
    if not os.path.exists(obj):
        pytest.skip(f"{name} is not built (__graft_entry__.build())")
    if not all(os.path.exists(f"{LLVM}/{t}") for t in ("llvm-objcopy", "clang-offload-bundler", "llvm-objdump")):
        pytest.skip("ROCm LLVM tools are not installed")
    dis = _disassemble(obj, tmp_path)
    if dis is None:
        return
    bad = sorted({m.group(0) for m in SCALAR_WRITE.finditer(dis)})
    assert not bad, f"{name}: scalar-memory writes {bad}"
    bad = sorted({m.group(0) for m in PACKED_F32.finditer(dis)})
    assert not bad, f"{name}: packed fp32 operations {bad}"
    if "kernels" in name:
        assert "v_mfma" in dis, f"{name}: no MFMA instruction found; is this the kernel object?"
