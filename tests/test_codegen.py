"""The built library's gfx950 code, on the CPU: no barrier sits in a loop
that exits by narrowing exec, no kernel spills vector registers to scratch,
and no kernel reaches memory through flat (generic address space)
instructions.  A flat access also counts
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


# ---------------------------------------------------------------------------
# Barriers and divergent loops.  A loop whose exit the compiler takes for
# divergent is laid out as a loop that ends by narrowing exec: the lanes that
# leave wait, masked off, while the others run the next round.  A workgroup
# barrier inside such a loop then completes with some lanes of a wave still
# in the previous round, and the others read what those lanes have not yet
# written to LDS.  (A form of the long-bag pass whose loop control came from
# LDS without readfirstlane livelocked this way: after a bag's last segment,
# every thread but thread 0 re-entered the loop and read a stale entry word.)
# Every kernel's loops around barriers must be controlled by wave-uniform
# values; this checks the compiled code for it.

SOURCES = ["eb_forward.hip", "eb_backward.hip", "eb_fm.hip", "eb_seq.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _device_asm(src, out):
    from paper_2609_30656_amd import build
    flags = [f for f in build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    return subprocess.Popen([HIPCC, *flags, "--cuda-device-only", "-S", "-I", build.INCLUDE, "-I", build.CSRC,
                             os.path.join(build.CSRC, src), "-o", str(out)],
                            stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)


def barriers_in_divergent_loops(asm):
    """{kernel: (barriers, barriers inside a loop that exits by narrowing exec)}
    from compiler assembly (-S), whose block comments name each block's loops."""
    out = {}
    lines = asm.split("\n")
    i = 0
    while i < len(lines):
        m = re.match(r"^(_Z\S+):\s*;\s*@", lines[i])
        if not m:
            i += 1
            continue
        name, j = m.group(1), i + 1
        while j < len(lines) and not lines[j].startswith(".Lfunc_end"):
            j += 1
        blocks = []  # [label, comment, instructions]
        for line in lines[i + 1:j]:
            bm = re.match(r"^(\.LBB\d+_\d+|; %bb\.\d+):\s*(;.*)?$", line)
            if bm:
                blocks.append([bm.group(1).replace(".L", ""), bm.group(2) or "", []])
            elif blocks and re.match(r"^\s+;", line) and not blocks[-1][2]:
                blocks[-1][1] += " " + line.strip()
            elif blocks:
                blocks[-1][2].append(line.strip())
        parent_of, divergent, where = {}, set(), []
        for label, comment, ins in blocks:
            parents = set(re.findall(r"Parent Loop (BB\d+_\d+)", comment))
            if "This Loop Header" in comment or "This Inner Loop Header" in comment:
                inner = label
                parent_of[label] = parents
            else:
                h = re.findall(r"in Loop: Header=(BB\d+_\d+)", comment)
                inner = h[0] if h else None
            if inner and any(s.startswith("s_andn2_b64 exec, exec") for s in ins):
                divergent.add(inner)
            where += [{inner} | parents if inner else parents for s in ins if s.startswith("s_barrier")]

        def enclosing(loops):
            seen, todo = set(loops), list(loops)
            while todo:
                for p in parent_of.get(todo.pop(), ()):
                    if p not in seen:
                        seen.add(p)
                        todo.append(p)
            return seen

        out[name] = (len(where), sum(1 for w in where if enclosing(w) & divergent))
        i = j
    return out


@pytest.fixture(scope="module")
def device_asm(tmp_path_factory):
    """{source: compiler assembly (-S) of its gfx950 device code}, compiled once."""
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not found")
    d = tmp_path_factory.mktemp("asm")
    procs = {src: _device_asm(src, d / (src + ".s")) for src in SOURCES}
    out = {}
    for src, p in procs.items():
        assert p.wait(timeout=600) == 0, f"{src}: hipcc failed"
        out[src] = (d / (src + ".s")).read_text()
    return out


def test_no_barrier_in_a_divergent_loop(device_asm):
    total = 0
    for src, text in device_asm.items():
        found = barriers_in_divergent_loops(text)
        assert found, f"{src}: no kernel found in the assembly"
        for name, (nbar, bad) in found.items():
            total += nbar
            assert bad == 0, f"{src}: {name}: {bad} of {nbar} barriers inside a loop that exits by narrowing exec"
    assert total > 50  # the long-bag pass, the sort and the keys kernel hold barriers in loops


def test_divergent_loop_check_flags_a_barrier_in_one():
    # the check itself, on a hand-made listing: loop BB0_1 ends by narrowing
    # exec and holds a barrier
    asm = "\n".join([
        "_Zkern:                                 ; @_Zkern",
        "; %bb.0:",
        "\ts_mov_b64 s[0:1], 0",
        ".LBB0_1:                                ; =>This Inner Loop Header: Depth=1",
        "\ts_barrier",
        "\tv_cmp_le_i32_e32 vcc, s2, v0",
        "\ts_or_b64 s[0:1], vcc, s[0:1]",
        "\ts_andn2_b64 exec, exec, s[0:1]",
        "\ts_cbranch_execnz .LBB0_1",
        "; %bb.2:",
        "\ts_endpgm",
        ".Lfunc_end0:",
    ])
    assert barriers_in_divergent_loops(asm) == {"_Zkern": (1, 1)}
    uniform = asm.replace("\ts_andn2_b64 exec, exec, s[0:1]", "\ts_cmp_lg_u32 s3, 0")
    assert barriers_in_divergent_loops(uniform) == {"_Zkern": (1, 0)}


# ---------------------------------------------------------------------------
# Register spills.  A kernel that spills vector registers keeps values in
# scratch memory: one more round trip inside loops that are meant to be bound
# by the row loads alone.  Every kernel is sized (batch depth, the occupancy
# each asks the compiler for) to fit its vector registers; this keeps it so.
# (Scalar registers that overflow go to lanes of vector registers, not to
# memory, so they are reported but allowed.)

def kernel_spills(asm):
    """{kernel: (vgpr_count, vgpr_spill_count, sgpr_spill_count, scratch bytes
    per lane)} from the code object metadata in compiler assembly."""
    out = {}
    for block in asm.split("  - .agpr_count:")[1:]:
        f = {k: re.search(r"\." + k + r":\s+(\S+)", block) for k in
             ("name", "vgpr_count", "vgpr_spill_count", "sgpr_spill_count", "private_segment_fixed_size")}
        if all(f.values()):
            out[f["name"].group(1)] = tuple(int(f[k].group(1)) for k in
                                            ("vgpr_count", "vgpr_spill_count", "sgpr_spill_count",
                                             "private_segment_fixed_size"))
    return out


def test_no_kernel_spills_vector_registers(device_asm):
    total = 0
    for src, text in device_asm.items():
        found = kernel_spills(text)
        assert found, f"{src}: no kernel metadata in the assembly"
        total += len(found)
        spilling = {k: v for k, v in found.items() if v[1] or v[3]}
        assert not spilling, f"{src}: kernels with vector spills or scratch (vgprs, vgpr spills, sgpr spills, " \
                             f"scratch bytes): {spilling}"
    assert total > 50


def test_spill_check_reads_the_metadata():
    block = ("  - .agpr_count:     0\n    .name:           _Zk\n    .private_segment_fixed_size: 16\n"
             "    .sgpr_spill_count: 0\n    .vgpr_count:     72\n    .vgpr_spill_count: 3\n")
    assert kernel_spills("amdhsa.kernels:\n" + block) == {"_Zk": (72, 3, 0, 16)}
