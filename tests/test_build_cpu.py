"""The built library's device code, inspected on the CPU: it contains no
packed-fp32 instructions (the device pass disables their formation) and no
kernel uses scratch memory (a spill would slow every role sharing the
kernel).  Reads only the code object built here from this repository's
sources."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2406_11016_amd import binding

LLVM = "/opt/rocm/lib/llvm/bin"


def _tool(name):
    path = os.path.join(LLVM, name)
    if not os.path.exists(path):
        pytest.skip(f"{name} not available")
    return path


@pytest.fixture(scope="module")
def code_object(tmp_path_factory):
    if not os.path.exists(binding.LIB_PATH):
        pytest.fail("libspec_verify.so not built; run __graft_entry__.build()")
    d = tmp_path_factory.mktemp("co")
    fb, co = str(d / "fb.bin"), str(d / "co.o")
    subprocess.run([_tool("llvm-objcopy"), "--dump-section", f".hip_fatbin={fb}", binding.LIB_PATH, str(d / "x")],
                   check=True, capture_output=True)
    subprocess.run([_tool("clang-offload-bundler"), "-type=o", "-targets=hipv4-amdgcn-amd-amdhsa--gfx950",
                    f"-input={fb}", f"-output={co}", "-unbundle"], check=True, capture_output=True)
    return co


def test_no_packed_fp32_instructions(code_object):
    dis = subprocess.run([_tool("llvm-objdump"), "-d", code_object], check=True, capture_output=True,
                         text=True).stdout
    assert "s_endpgm" in dis
    packed = re.findall(r"\bv_pk_(?:add|mul|fma)_f32\b", dis)
    assert not packed, f"{len(packed)} packed-fp32 instructions in the device code"


def test_no_kernel_uses_scratch(code_object):
    notes = subprocess.run([_tool("llvm-readelf"), "--notes", code_object], check=True, capture_output=True,
                           text=True).stdout
    names = re.findall(r"\.name:\s+(_Z\S+)", notes)
    scratch = [int(x) for x in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", notes)]
    assert len(names) == len(scratch) and any("verify_kernel" in n for n in names)
    spills = {n: s for n, s in zip(names, scratch) if s}
    assert not spills, spills
