"""The build's check of the hand-written memory instructions (isa_check.py):
hazards planted in small assembly listings are found, their guarded forms
pass, and the projection kernel's device assembly has none."""
import os
import shutil

import pytest

from paper_1805_09863_amd import _build, isa_check


def kernel(body: str, name: str = "_Z1kv") -> str:
    return (f"\t.type\t{name},@function\n{name}:  ; @{name}\n; %bb.0:\n" + body +
            "\ts_endpgm\n.Lfunc_end0:\n\t.size\t" + name + ", .Lfunc_end0-" + name + "\n")


def asm(*lines: str) -> str:
    return ";;#ASMSTART\n" + "".join("\t" + x + "\n" for x in lines) + ";;#ASMEND\n"


def ins(*lines: str) -> str:
    return "".join("\t" + x + "\n" for x in lines)


RESTORE = ins("v_readlane_b32 s8, v172, 14", "v_readlane_b32 s9, v172, 15")


def test_restored_base_right_before_load():
    bad = isa_check.check(kernel(RESTORE + asm("global_load_dword v15, v60, s[8:9]")))
    assert len(bad) == 1 and "0 wait state" in bad[0] and "v_readlane_b32 s9" in bad[0]


@pytest.mark.parametrize("nop,ok", [(0, False), (3, False), (4, True), (7, True)])
def test_wait_states_counted(nop, ok):
    body = RESTORE + ins(f"s_nop {nop}") + asm("global_load_dword v15, v60, s[8:9]")
    assert (isa_check.check(kernel(body)) == []) == ok


def test_other_instructions_count_as_wait_states():
    filler = ins(*["v_mov_b32 v1, v2"] * 4)
    assert isa_check.check(kernel(RESTORE + filler + asm("global_load_dword v15, v60, s[8:9]")))
    filler = ins(*["v_mov_b32 v1, v2"] * 5)       # 5 instructions between the write of s9 and the load
    assert isa_check.check(kernel(RESTORE + filler + asm("global_load_dword v15, v60, s[8:9]"))) == []


def test_scalar_copy_guard_passes():
    body = RESTORE + asm("s_mov_b64 s[0:1], s[8:9]", "global_load_dword v15, v60, s[0:1]")
    assert isa_check.check(kernel(body)) == []


def test_other_registers_and_vop3b_carry():
    assert isa_check.check(kernel(RESTORE + asm("global_load_dword v15, v60, s[10:11]"))) == []
    carry = ins("v_add_co_u32_e64 v1, s[10:11], v2, v3")
    assert isa_check.check(kernel(carry + asm("global_load_dword v15, v60, s[10:11]")))


def test_hazard_across_a_branch():
    # the write sits before a branch to the load's label; the fall-through
    # path in between is padded, the branch path is not
    body = (ins("v_readfirstlane_b32 s4, v0", "s_cbranch_scc1 .LBB0_2") + ins(*["s_nop 7"] * 2) +
            ".LBB0_2:\n" + asm("global_load_dword v1, v2, s[4:5]"))
    bad = isa_check.check(kernel(body))
    assert len(bad) == 1 and "1 wait state" in bad[0]


def test_unconditional_branch_ends_fall_through():
    body = (ins("v_readfirstlane_b32 s4, v0", "s_branch .LBB0_3") + ".LBB0_2:\n" +
            asm("global_load_dword v1, v2, s[4:5]") + ".LBB0_3:\n" + ins("s_nop 0"))
    assert isa_check.check(kernel(body)) == []


def test_m0_rules():
    dma = asm("global_load_lds_dwordx4 v1, s[4:5] offset:0")
    set_m0 = asm("s_mov_b32 m0, s6", "s_nop 0")
    assert isa_check.check(kernel(set_m0 + dma)) == []
    bad = isa_check.check(kernel(set_m0 + ins("s_mov_b32 m0, -1") + dma))
    assert len(bad) == 1 and "compiler code writes M0" in bad[0]
    bad = isa_check.check(kernel(asm("s_mov_b32 m0, s6") + dma))
    assert len(bad) == 1 and "no wait state" in bad[0]


def test_kernels_are_separate():
    two = kernel(RESTORE, "_Z1av") + kernel(asm("global_load_dword v1, v2, s[8:9]"), "_Z1bv")
    assert isa_check.check(two) == []


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not installed")
def test_projection_kernel_assembly_has_no_hazard(tmp_path, monkeypatch):
    """The kernel that faulted when its epilogue's scalar base was restored
    right before an inline-assembly load: every instantiation's device
    assembly is free of the hazard."""
    monkeypatch.setattr(_build, "OBJDIR", str(tmp_path))
    path = _build._device_asm(_build._hipcc(), os.path.join(_build.CSRC, "k1_wide.hip"))
    text = open(path).read()
    assert len(isa_check.parse(text)) >= 6
    assert isa_check.check(text) == []
