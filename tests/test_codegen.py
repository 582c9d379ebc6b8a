"""The built library's gfx950 code, on the CPU: no kernel reaches memory
through flat (generic address space) instructions.  A flat access also counts
against the LDS counter, so a wait for a cross-lane shuffle would wait for
it too; every table row, optimizer state and partial sum is addressed in the
global address space instead.  The code objects are unbundled from libeb.so
(built here) into a temporary directory and disassembled."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_30656_amd", "libeb.so")
OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"


def _gfx950_objects(tmp_path):
    if not os.path.exists(LIB):
        pytest.skip("libeb.so is not built")
    if not os.path.exists(OBJDUMP):
        pytest.skip("llvm-objdump not found")
    lib = tmp_path / "libeb.so"
    shutil.copy(LIB, lib)
    subprocess.run([OBJDUMP, "--offloading", str(lib)], cwd=tmp_path, check=True, capture_output=True,
                   timeout=120)
    objs = sorted(p for p in tmp_path.iterdir() if p.name.endswith("gfx950"))
    assert objs, "no gfx950 code object in libeb.so"
    return objs


def test_no_flat_memory_instructions(tmp_path):
    objs = _gfx950_objects(tmp_path)
    mem = flat = 0
    for o in objs:
        text = subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", str(o)], check=True, capture_output=True,
                              text=True, timeout=300).stdout
        mem += len(re.findall(r"^\s+(?:global|buffer)_(?:load|store|atomic)", text, re.M))
        bad = re.findall(r"^\s+(flat_\w+)", text, re.M)
        flat += len(bad)
        assert not bad, f"{o.name}: {len(bad)} flat memory instructions, e.g. {bad[:3]}"
    assert mem > 1000  # the disassembly really holds the kernels
    assert flat == 0
