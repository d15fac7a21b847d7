"""Helpers for tests that inspect the library's own built gfx950 code objects (built here from
the sources under paper_2407_09577_amd/csrc) with the ROCm LLVM tools."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "paper_2407_09577_amd", "_build")
LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"


def code_object(source, tmp_path):
    """Path of the gfx950 code object unbundled from the built object of csrc/<source>."""
    for tool in ("clang-offload-bundler", "llvm-objdump", "llvm-readelf"):
        if not os.path.exists(os.path.join(LLVM, tool)):
            pytest.skip(f"{tool} not installed")
    if shutil.which("objcopy") is None:
        pytest.skip("objcopy not installed")
    obj = os.path.join(BUILD, source + ".o")
    if not os.path.exists(obj):
        pytest.skip("library not built")
    fat, co = tmp_path / (source + ".fat"), tmp_path / (source + ".co")
    subprocess.run(["objcopy", f"--dump-section=.hip_fatbin={fat}", obj], check=True, capture_output=True)
    subprocess.run([os.path.join(LLVM, "clang-offload-bundler"), "--unbundle", "--type=o", f"--input={fat}",
                    f"--targets={TARGET}", f"--output={co}"], check=True, capture_output=True)
    return co


def disassemble(source, tmp_path):
    """Instruction text of every kernel in the code object (address and encoding dropped)."""
    out = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", "--mcpu=gfx950", str(code_object(source, tmp_path))],
                         check=True, capture_output=True, text=True).stdout
    return [ln.split("//")[0].strip() for ln in out.splitlines() if ln.startswith("\t")]


def kernel_resources(source, tmp_path):
    """{mangled kernel name: {field: int}} from the code object's kernel metadata."""
    out = subprocess.run([os.path.join(LLVM, "llvm-readelf"), "--notes", str(code_object(source, tmp_path))],
                         check=True, capture_output=True, text=True).stdout
    res = {}
    for chunk in re.split(r"\n\s+- \.", out):
        m = re.search(r"\.name:\s+(\S+)", chunk)
        if not m or ".private_segment_fixed_size" not in chunk:
            continue
        fields = {k: int(v) for k, v in re.findall(r"\.(\w+):\s+(\d+)\s*$", chunk, flags=re.M)}
        res[m.group(1)] = fields
    return res


def template_args(mangled):
    """Integer and bool template arguments of a mangled kernel name, in order."""
    m = re.search(r"kernelI((?:L[ib]\d+E)+)E", mangled)
    return [int(x) for x in re.findall(r"L[ib](\d+)E", m.group(1))] if m else []
