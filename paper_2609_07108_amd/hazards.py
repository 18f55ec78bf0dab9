"""Static check of the gfx950 hazards that the compiler cannot pad for us.

The ring kernels issue some MFMAs and every direct global-to-LDS load as
inline assembly.  The compiler does not look inside those statements, so the
wait states that the hardware requires around them (and that the compiler
inserts for its own instructions) are the kernels' responsibility.  This
module reads the device assembly that the build produces (``-save-temps``)
and checks, along every control-flow path, the rules below.  ``build()``
runs it on every source and refuses a library that breaks one.

Rules (wait states: one per issued instruction, N + 1 for ``s_nop N``):

R1  An MFMA result (32x32x16, eight passes) may not be read or overwritten by
    any other instruction within 12 wait states, except by an MFMA that
    accumulates into exactly the same registers (its C operand and result are
    the registers written).  This covers vector-ALU reads and writes, LDS and
    memory instructions, accumulation-register moves, and MFMAs that take the
    result as an A or B operand.
R2  A register written by a vector-ALU instruction may not be read by an
    inline-assembly MFMA within 2 wait states.
R3  M0 written by a scalar instruction may not be read by a direct
    global-to-LDS load (``global_load_lds_*``, ``buffer_load_* ... lds``)
    within 1 wait state.
"""

from __future__ import annotations

import re
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Set, Tuple

MFMA_RESULT_WAIT = 12
VALU_TO_MFMA_WAIT = 2
M0_TO_LDS_DMA_WAIT = 1

_REG = re.compile(r"\b([va])(?:\[(\d+):(\d+)\]|(\d+)\b)")
_LABEL = re.compile(r"^([.\w$]+):")


@dataclass
class Instr:
    line: int            # line number in the assembly file (1-based)
    text: str
    op: str
    operands: List[str]
    inline: bool         # inside an inline-assembly block
    label_targets: List[str] = field(default_factory=list)

    def regs(self, idx: Optional[int] = None) -> Set[Tuple[str, int]]:
        ops = self.operands if idx is None else self.operands[idx:idx + 1]
        out = set()
        for o in ops:
            for m in _REG.finditer(o):
                cls = m.group(1)
                if m.group(4) is not None:
                    out.add((cls, int(m.group(4))))
                else:
                    out.update((cls, r) for r in range(int(m.group(2)), int(m.group(3)) + 1))
        return out

    def wait_states(self) -> int:
        if self.op == "s_nop":
            return int(self.operands[0], 0) + 1 if self.operands else 1
        return 1

    @property
    def is_mfma(self) -> bool:
        return self.op.startswith("v_mfma")

    @property
    def is_valu(self) -> bool:
        return self.op.startswith("v_") and not self.is_mfma

    def valu_defs(self) -> Set[Tuple[str, int]]:
        """Registers written by a vector-ALU instruction (its first operand)."""
        return self.regs(0) if self.is_valu and self.operands else set()

    @property
    def is_lds_dma(self) -> bool:
        return self.op.startswith("global_load_lds") or (self.op.startswith("buffer_load") and
                                                         any(o.strip() == "lds" for o in self.operands))

    @property
    def writes_m0(self) -> bool:
        return self.op.startswith("s_") and bool(self.operands) and self.operands[0].strip() == "m0"


@dataclass
class Function:
    name: str
    instrs: List[Instr]
    labels: Dict[str, int]   # label -> index of the next instruction

    def succ(self, i: int) -> List[int]:
        ins = self.instrs[i]
        out = []
        if ins.op in ("s_endpgm", "s_setpc_b64"):
            return out
        if ins.op != "s_branch" and i + 1 < len(self.instrs):
            out.append(i + 1)
        for t in ins.label_targets:
            if t in self.labels and self.labels[t] < len(self.instrs):
                out.append(self.labels[t])
        return out


def parse(asm: str) -> List[Function]:
    funcs: List[Function] = []
    cur: Optional[Function] = None
    inline = False
    pending: List[str] = []
    for n, raw in enumerate(asm.splitlines(), 1):
        line = raw.split(";")[0].rstrip() if not raw.lstrip().startswith(";;#ASM") else raw.strip()
        s = raw.strip()
        if s.startswith(";;#ASMSTART"):
            inline = True
            continue
        if s.startswith(";;#ASMEND"):
            inline = False
            continue
        if s.startswith(".type") and "@function" in s:
            name = s.split()[1].split(",")[0]
            cur = Function(name, [], {})
            funcs.append(cur)
            pending = []
            continue
        if cur is None:
            continue
        if s.startswith(".Lfunc_end"):
            cur = None
            continue
        m = _LABEL.match(line.strip())
        if m:
            cur.labels[m.group(1)] = len(cur.instrs)
            continue
        body = line.strip()
        if not body or body.startswith("."):
            continue
        parts = body.split(None, 1)
        op = parts[0]
        operands = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
        targets = [o for o in operands if o.startswith(".L")] if op.startswith(("s_branch", "s_cbranch")) else []
        cur.instrs.append(Instr(n, body, op, operands, inline, targets))
    return funcs


def _forward_window(f: Function, start: int, budget: int):
    """Instructions reachable from `start` (exclusive) while fewer than
    `budget` wait states have passed: yields (index, wait states before it)."""
    seen: Dict[int, int] = {}
    stack = [(s, 0) for s in f.succ(start)]
    while stack:
        i, w = stack.pop()
        if w >= budget or seen.get(i, -1) >= budget - w:
            continue
        seen[i] = budget - w
        yield i, w
        nw = w + f.instrs[i].wait_states()
        stack.extend((s, nw) for s in f.succ(i))


def _preds(f: Function) -> List[List[int]]:
    p: List[List[int]] = [[] for _ in f.instrs]
    for i in range(len(f.instrs)):
        for s in f.succ(i):
            p[s].append(i)
    return p


def _backward_window(f: Function, preds, start: int, budget: int):
    seen: Dict[int, int] = {}
    stack = [(q, 0) for q in preds[start]]
    while stack:
        i, w = stack.pop()
        if w >= budget or seen.get(i, -1) >= budget - w:
            continue
        seen[i] = budget - w
        yield i, w
        nw = w + f.instrs[i].wait_states()
        stack.extend((q, nw) for q in preds[i])


def check_function(f: Function) -> List[str]:
    errs = []
    preds = None
    for i, ins in enumerate(f.instrs):
        if ins.is_mfma and ins.operands:
            dst = ins.regs(0)
            for j, w in _forward_window(f, i, MFMA_RESULT_WAIT):
                other = f.instrs[j]
                if not (other.regs() & dst):
                    continue
                if other.is_mfma and other.regs(0) == dst and len(other.operands) > 3 and other.regs(3) == dst and \
                        not ((other.regs(1) | other.regs(2)) & dst):
                    continue  # accumulation chain into the same registers
                errs.append(f"{f.name}: R1 line {other.line} ({other.text}) touches the result of the MFMA at "
                            f"line {ins.line} after {w} wait states (needs {MFMA_RESULT_WAIT})")
        if ins.is_mfma and ins.inline:
            preds = preds or _preds(f)
            srcs = set()
            for k in (1, 2, 3):
                if k < len(ins.operands):
                    srcs |= ins.regs(k)
            for j, w in _backward_window(f, preds, i, VALU_TO_MFMA_WAIT):
                if f.instrs[j].valu_defs() & srcs:
                    errs.append(f"{f.name}: R2 line {ins.line} ({ins.text}) reads a register written by the "
                                f"vector ALU at line {f.instrs[j].line} after {w} wait states "
                                f"(needs {VALU_TO_MFMA_WAIT})")
        if ins.is_lds_dma:
            preds = preds or _preds(f)
            for j, w in _backward_window(f, preds, i, M0_TO_LDS_DMA_WAIT):
                if f.instrs[j].writes_m0:
                    errs.append(f"{f.name}: R3 line {ins.line} ({ins.text}) reads M0 written at line "
                                f"{f.instrs[j].line} after {w} wait states (needs {M0_TO_LDS_DMA_WAIT})")
    return errs


def check_asm(asm: str) -> List[str]:
    errs = []
    for f in parse(asm):
        errs.extend(check_function(f))
    return errs


def check_file(path: str) -> List[str]:
    with open(path) as fh:
        return [f"{path}: {e}" for e in check_asm(fh.read())]
