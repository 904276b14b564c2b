"""Layout of the node-per-wave layer's leaf tables in the built library (CPU).

The node-per-wave LUT kernel (csrc/lut_jump.hip) evaluates byte t of a node's
table as the 3-input function g_t(x0, x1, x2) = T[8t + x0 + 2 x1 + 4 x2]
(Shannon expansion of Sec. 3's node on its three upper inputs) by jumping to a
prebuilt leaf: one v_bitop3_b32 whose 8-bit truth table is that byte,
followed by a jump to the next byte's leaf.  The prep kernel computes leaf
addresses as base + t * 3072 + byte * 12, so the tables must be exactly that
dense.  This test disassembles the gfx950 code objects of
libbitlogic.so and checks every one of the 8 x 256 leaves: the instruction
at each computed address, its truth table, its destination and source
registers, and the jump that follows.  The GPU parity tests check the
results; this pins the table layout the addresses assume without a GPU.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2602_07400_amd import bitlogic as bl

OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"
READELF = "/opt/rocm/llvm/bin/llvm-readelf"
LEAF_BYTES, TABLE_BYTES = 12, 256 * 12


def _code_objects(tmp_path):
    if not (os.path.exists(OBJDUMP) and os.path.exists(READELF)):
        pytest.skip("llvm-objdump not installed")
    lib = bl.library_path()
    if not os.path.exists(lib):
        pytest.skip("library not built")
    dst = tmp_path / "libbitlogic.so"
    shutil.copy(lib, dst)
    subprocess.run([OBJDUMP, "--offloading", str(dst)], check=True, capture_output=True,
                   cwd=tmp_path)
    objs = sorted(p for p in tmp_path.iterdir() if "amdgcn" in p.name and "gfx950" in p.name)
    assert objs, "no gfx950 code object in the library"
    return objs


def _disassemble(obj):
    out = subprocess.run([OBJDUMP, "-d", str(obj)], check=True, capture_output=True,
                         text=True).stdout
    labels, ins = {}, {}
    for line in out.splitlines():
        m = re.match(r"^([0-9a-f]{16}) <(.*)>:", line)
        if m:
            labels[m.group(2)] = int(m.group(1), 16)
            continue
        m = re.match(r"^\s+(\S.*?)\s+// ([0-9A-F]{12}):", line)
        if m:
            ins[int(m.group(2), 16)] = m.group(1)
    return labels, ins


def _kernel_registers(obj):
    notes = subprocess.run([READELF, "--notes", str(obj)], check=True, capture_output=True,
                           text=True).stdout
    regs, name = {}, None
    for line in notes.splitlines():
        m = re.match(r"\s+\.name:\s+(\S+)", line)
        if m:
            name = m.group(1)
            regs[name] = {}
            continue
        m = re.match(r"\s+\.(sgpr_count|vgpr_count):\s+(\d+)", line)
        if m and name:
            regs[name][m.group(1)] = int(m.group(2))
    return regs


def test_leaf_tables_are_dense_and_correct(tmp_path):
    found = []
    for obj in _code_objects(tmp_path):
        labels, ins = _disassemble(obj)
        if "bl_jump_leaves" in labels:
            found.append((obj, labels, ins))
    assert len(found) == 1, "the leaf tables must be assembled exactly once"
    obj, labels, ins = found[0]
    base = labels["bl_jump_leaves"]
    for t in range(8):
        nxt = f"s_setpc_b64 s[{66 + 2 * t}:{67 + 2 * t}]" if t < 7 else "s_setpc_b64 s[80:81]"
        for b in range(256):
            a = base + t * TABLE_BYTES + b * LEAF_BYTES
            op = ins.get(a, "")
            m = re.match(r"v_bitop3_b32 v(\d+), v16, v15, v14(?: bitop3:(\S+))?$", op)
            assert m, f"leaf ({t}, {b:#x}) at {a:#x}: {op!r}"
            assert int(m.group(1)) == 20 + t, f"leaf ({t}, {b:#x}) writes v{m.group(1)}"
            tt = int(m.group(2), 0) if m.group(2) else 0
            assert tt == b, f"leaf ({t}, {b:#x}) has truth table {tt:#x}"
            assert ins.get(a + 8, "") == nxt, f"leaf ({t}, {b:#x}) continues with {ins.get(a + 8)!r}"


def test_layer_kernel_allocates_the_leaf_registers(tmp_path):
    # the leaves write v20..v27 and jump through s[66:81]: the layer kernel that
    # runs them must own those registers
    for obj in _code_objects(tmp_path):
        regs = _kernel_registers(obj)
        names = [n for n in regs if "k_jump_layer" in n]
        if names:
            assert len(names) == 1
            r = regs[names[0]]
            assert r["vgpr_count"] >= 28, r
            assert r["sgpr_count"] >= 82, r
            return
    pytest.fail("k_jump_layer not found")


def test_truth_table_operand_order():
    # v_bitop3_b32 D, S0, S1, S2 with table TT gives bit TT[4 S0 + 2 S1 + S2]
    # (the multiplexer 0xCA = S0 ? S1 : S2 is one instance).  A leaf passes
    # (x2, x1, x0), so its index is x0 + 2 x1 + 4 x2 = the address of entry
    # 8t + ... within byte t, i.e. the leaf of byte value B computes B[a].
    def bitop3(tt, s0, s1, s2):
        return (tt >> (4 * s0 + 2 * s1 + s2)) & 1

    for s0 in (0, 1):
        for s1 in (0, 1):
            for s2 in (0, 1):
                assert bitop3(0xCA, s0, s1, s2) == (s1 if s0 else s2)
    for B in (0x00, 0xFF, 0x96, 0xE8, 0x5A, 0x01, 0x80):
        for a in range(8):
            x0, x1, x2 = a & 1, (a >> 1) & 1, (a >> 2) & 1
            assert bitop3(B, x2, x1, x0) == (B >> a) & 1
