"""The selection walk enters its block of 16 depth steps by a computed jump
(PC + e * step size).  These checks run on the gfx950 code object that the
library's own flags produce, without a GPU: every entry e in 0..15 of every
copy of the block must be the first instruction of step e, even steps must
test one lane set's depth register and odd steps the other's, and the
block's back-edge must move both down by 16 and return to step 0.  A wrong entry would execute from the middle
of an instruction, so this is checked on every build rather than on the GPU.
"""
import os
import re
import shutil
import subprocess

import pytest

import paper_2602_06502_amd._build as B

OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"


def _disassemble(tmp_path):
    if not os.path.exists(B.HIPCC) or not os.path.exists(OBJDUMP):
        pytest.skip("ROCm compiler tools not installed")
    src = os.path.join(B.CSRC, "dm_select.hip")
    obj = str(tmp_path / "dm_select_gfx950.o")
    cmd = [B.HIPCC, *B.FLAGS, "--cuda-device-only", "--no-gpu-bundle-output", "-c", src, "-o", obj]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    out = subprocess.run([OBJDUMP, "-d", "--no-show-raw-insn", obj], stdout=subprocess.PIPE,
                         text=True, check=True).stdout
    ins = []
    for line in out.splitlines():
        m = re.match(r"\s+(\S.*?)\s*//\s*([0-9A-Fa-f]+):", line)
        if m:
            ins.append((int(m.group(2), 16), m.group(1).strip()))
    return ins


def test_walk_entries_land_on_step_starts(tmp_path):
    ins = _disassemble(tmp_path)
    at = {a: i for i, (a, _) in enumerate(ins)}
    lit = r"(0x[0-9a-f]+|\d+)"
    blocks = 0
    for i, (_, text) in enumerate(ins):
        if text != "s_getpc_b64 s[96:97]":
            continue
        blocks += 1
        # the window's control word e | (passes - 1) << 4 is read just before
        assert re.fullmatch(r"v_readfirstlane_b32 s99, v\d+", ins[i - 1][1]), ins[i - 1]
        pc = ins[i + 1][0]  # s_getpc_b64 yields the address of the next instruction
        assert ins[i + 1][1] == "s_and_b32 s98, s99, 15", ins[i + 1]  # e < 16
        mul = re.fullmatch(r"s_mul_i32 s98, s98, " + lit, ins[i + 2][1])
        add = re.fullmatch(r"s_add_u32 s98, s98, " + lit, ins[i + 3][1])
        assert mul and add, (ins[i + 2], ins[i + 3])
        assert ins[i + 4][1] == "s_add_u32 s96, s96, s98"
        assert ins[i + 5][1] == "s_addc_u32 s97, s97, 0"
        # passes - 1 = bits 4..5 of the control word: at most four passes
        assert ins[i + 6][1] == "s_bfe_u32 s99, s99, 0x20004", ins[i + 6]
        assert ins[i + 7][1] == "s_setpc_b64 s[96:97]"
        step, off = int(mul.group(1), 0), int(add.group(1), 0)
        assert pc + off == ins[i + 8][0], "entry 0 is not the instruction after the jump"
        rel = {0: set(), 1: set()}  # the rel register of each lane set
        for e in range(16):
            tgt = pc + e * step + off
            assert tgt in at, f"entry {e} lands inside an instruction"
            j = at[tgt]
            assert ins[j][1].startswith("ds_read_b32"), ins[j]
            assert ins[j + 1][1].startswith("ds_read_b32"), ins[j + 1]
            m = re.fullmatch(r"v_cmp_eq_u32_e64 s\[\d+:\d+\], (\d+), (v\d+)", ins[j + 2][1])
            assert m and int(m.group(1)) == e, (e, ins[j + 2])
            rel[e & 1].add(m.group(2))
        # even steps test set A's rel, odd steps set B's
        assert len(rel[0]) == 1 and len(rel[1]) == 1 and rel[0] != rel[1], rel
        j = at[pc + 16 * step + off]
        # the back-edge moves both sets' rel down by 16
        backs = set()
        for k in (j, j + 1):
            m = re.fullmatch(r"v_add_u32_e32 (v\d+), -16, \1", ins[k][1])
            assert m, ins[k]
            backs.add(m.group(1))
        assert backs == rel[0] | rel[1], (backs, rel)
        assert ins[j + 2][1] == "s_sub_u32 s99, s99, 1", ins[j + 2]
        br_addr, br = ins[j + 3]
        assert br.startswith("s_cbranch_scc0"), br
        simm = int(br.split()[-1], 0)
        simm = simm - 65536 if simm >= 32768 else simm
        assert br_addr + 4 + 4 * simm == pc + off, "back-edge does not return to step 0"
    # one copy per record slot of the unrolled window loop
    src = open(os.path.join(B.CSRC, "dm_select.hip")).read()
    prefetch = int(re.search(r"constexpr int kPrefetch = (\d+);", src).group(1))
    assert blocks == prefetch

