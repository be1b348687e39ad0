"""Build-time check of two hazards that the compiler does not handle for the
hand-written (inline-assembly) memory instructions of the projection kernel.

1. A vector memory instruction that reads an SGPR needs 5 wait states after a
   VALU instruction that wrote that SGPR (v_readlane / v_readfirstlane, the
   carry-out of v_add_co and the like, a v_cmp's mask).  The compiler pads its
   own instructions; for an inline-assembly load it does not, and when it
   spills the load's base pair and restores it (v_readlane) right before the
   load, the load reads a stale base.
2. An inline-assembly LDS DMA (global_load_lds_*) reads M0, which an earlier
   inline-assembly statement set; the compiler does not track M0 across
   inline assembly, so in a kernel with such DMAs no compiler-generated
   instruction may write M0, and each inline-assembly M0 write is followed by
   an s_nop (a scalar M0 write needs one wait state before an LDS DMA).

The check reads the device assembly (``hipcc --cuda-device-only -S``).  For
(1) it walks every control-flow path backwards from each vector memory
instruction (fall-through and branches to its labels), counting wait states
(one per instruction, N+1 per s_nop N).  It runs over every vector memory instruction,
the compiler's included, so a wait-state model that disagrees with the
compiler's shows up as a failure too.
"""
from __future__ import annotations

import re
from dataclasses import dataclass, field

VMEM_PREFIX = ("global_", "buffer_", "scratch_", "flat_")
# VOP3b forms: the second operand is an SGPR (pair) written by the VALU
VOP3B = ("v_add_co_", "v_sub_co_", "v_subrev_co_", "v_addc_co_", "v_subb_co_", "v_subbrev_co_",
         "v_div_scale_", "v_mad_u64_u32", "v_mad_i64_i32")
SGPR_VMEM_WAIT = 5


@dataclass
class Inst:
    op: str
    ops: list[str]
    text: str
    in_asm: bool
    labels: list[str] = field(default_factory=list)   # labels right before this instruction


def _sgprs(tok: str) -> set[int | str]:
    tok = tok.strip().split()[0] if tok.strip() else ""
    m = re.fullmatch(r"s\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.fullmatch(r"s(\d+)", tok)
    if m:
        return {int(m.group(1))}
    if tok in ("vcc", "vcc_lo", "vcc_hi", "m0", "exec", "exec_lo", "exec_hi"):
        return {tok.split("_")[0]}
    return set()


def parse(asm: str) -> dict[str, list[Inst]]:
    """Kernels of an assembly file: name -> instructions in program order."""
    kernels: dict[str, list[Inst]] = {}
    funcs = set(re.findall(r"\.type\s+([\w.$]+),@function", asm))
    cur: list[Inst] | None = None
    in_asm = False
    pending: list[str] = []
    for line in asm.split("\n"):
        t = line.strip()
        if t.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if t.startswith(";;#ASMEND"):
            in_asm = False
            continue
        t = t.split(";")[0].strip()
        if not t or t.startswith("//"):
            continue
        m = re.fullmatch(r"([A-Za-z_.$][\w.$]*):", t)
        if m:
            name = m.group(1)
            if name in funcs:
                cur = kernels.setdefault(name, [])
                pending = []
            elif name.startswith(".Lfunc_end"):
                cur = None
            else:
                pending.append(name)
            continue
        if t.startswith(".") or cur is None:
            continue
        op, _, rest = t.partition(" ")
        ops = [o.strip() for o in rest.split(",")] if rest.strip() else []
        cur.append(Inst(op, ops, t, in_asm, pending))
        pending = []
    return kernels


def _valu_sgpr_writes(ins: Inst) -> set:
    if not ins.op.startswith("v_"):
        return set()
    w = set()
    if ins.ops:
        w |= _sgprs(ins.ops[0])
    if len(ins.ops) > 1 and ins.op.startswith(VOP3B):
        w |= _sgprs(ins.ops[1])
    if ins.op.startswith(("v_cmp_", "v_cmpx_")) and ins.op.endswith("_e32"):
        w.add("vcc")
    w.discard("exec")
    w.discard("m0")
    return w


def _wait_states(ins: Inst) -> int:
    if ins.op == "s_nop":
        return int(ins.ops[0], 0) + 1 if ins.ops else 1
    return 1


def _preds(insts: list[Inst], branches: dict[str, list[int]], i: int) -> list[int]:
    p = []
    if i > 0 and insts[i - 1].op not in ("s_branch", "s_endpgm", "s_setpc_b64"):
        p.append(i - 1)
    for lab in insts[i].labels:
        p.extend(branches.get(lab, []))
    return p


def check_kernel(insts: list[Inst]) -> list[str]:
    branches: dict[str, list[int]] = {}
    for i, ins in enumerate(insts):
        if ins.op.startswith(("s_branch", "s_cbranch")) and ins.ops:
            branches.setdefault(ins.ops[-1], []).append(i)
    bad = []
    for j, ins in enumerate(insts):
        if not ins.op.startswith(VMEM_PREFIX):
            continue
        reads = set()
        for o in ins.ops:
            reads |= _sgprs(o)
        reads.discard("m0")
        if reads:
            # backwards over every path until 5 wait states separate it from the load
            stack = [(p, 0) for p in _preds(insts, branches, j)]
            seen = set()
            while stack:
                i, ws = stack.pop()
                if (i, ws) in seen:
                    continue
                seen.add((i, ws))
                hit = _valu_sgpr_writes(insts[i]) & reads
                if hit:
                    bad.append(f"{ins.text!r} reads {sorted(map(str, hit))} {ws} wait state(s) after "
                               f"{insts[i].text!r}")
                    break
                ws2 = ws + _wait_states(insts[i])
                if ws2 < SGPR_VMEM_WAIT:
                    stack.extend((p, ws2) for p in _preds(insts, branches, i))
    # M0: written only by inline assembly (which then waits one state), so
    # that what an LDS DMA reads is what the source set; whether the right
    # inline-assembly write precedes each DMA is the source's logic
    m0_asm = [i for i, ins in enumerate(insts) if ins.in_asm and ins.ops and _sgprs(ins.ops[0]) == {"m0"}
              and not ins.op.startswith(VMEM_PREFIX)]
    if m0_asm or any(ins.in_asm and "_lds_" in ins.op for ins in insts):
        for i, ins in enumerate(insts):
            if ins.ops and _sgprs(ins.ops[0]) == {"m0"} and not ins.op.startswith(VMEM_PREFIX) and not ins.in_asm:
                bad.append(f"compiler code writes M0: {ins.text!r}")
        for i in m0_asm:
            if i + 1 >= len(insts) or insts[i + 1].op != "s_nop":
                bad.append(f"no wait state after {insts[i].text!r}")
    return bad


def check(asm: str) -> list[str]:
    """Every hazard found in an assembly file, as 'kernel: description'."""
    out = []
    for name, insts in parse(asm).items():
        out.extend(f"{name}: {b}" for b in check_kernel(insts))
    return out
