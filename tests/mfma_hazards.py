"""Static check of MFMA data hazards in gfx950 assembly.

The extend kernel issues its MFMAs from inline assembly, and the compiler
inserts no wait states around inline assembly, so the kernel keeps them by
itself (s_nop runs, instruction order).  This checker scans the assembly of
each kernel for the dependency rules that the hardware does not interlock,
counting wait states conservatively (one per instruction, N + 1 for s_nop N)
along every control-flow path, loops included.  The counts depend on the
instruction's pass count: v_mfma_f32_16x16x32_bf16 (16 cycles) and
v_mfma_f32_32x32x16_bf16 (32 cycles, 8 passes):

* VALU write of a register, then an MFMA reading it (A, B or C): 2.
* MFMA write of a register, then a VALU, LDS or memory instruction reading
  or writing it: 11 (16x16x32) or 12 (32x32x16; the compiler itself puts
  s_nop 11 after such an MFMA) -- the value is not there yet.
* MFMA write of a register, then an MFMA reading it as A or B: the same.
  (Reading it as C with the identical register range is the accumulation
  chain, which the hardware forwards.)
* MFMA read of its C operand, then a VALU, LDS or memory instruction writing
  that register: 7 (16x16x32) or 11 (32x32x16) -- the operand is read some
  passes after issue.

Used by tests/test_kernel_hazards.py; it reads text only.
"""
from __future__ import annotations

import re
from dataclasses import dataclass, field

VALU_MFMA = 2
MFMA_READ = 11
MFMA_SRCC_WAR = 7
# per-opcode (result-read, C-operand write-after-read) wait states
_WAITS = {"v_mfma_f32_32x32x16_bf16": (12, 11)}


def _waits(op: str) -> tuple[int, int]:
    return _WAITS.get(op, (MFMA_READ, MFMA_SRCC_WAR))

_REG = re.compile(r"^([va])(?:\[(\d+):(\d+)\]|(\d+))$")


def _regs(tok: str) -> frozenset:
    m = _REG.match(tok.strip())
    if not m:
        return frozenset()
    kind = m.group(1)
    if m.group(4) is not None:
        return frozenset({(kind, int(m.group(4)))})
    return frozenset((kind, r) for r in range(int(m.group(2)), int(m.group(3)) + 1))


@dataclass
class Ins:
    text: str
    op: str
    defs: frozenset = frozenset()
    uses: frozenset = frozenset()
    mfma: bool = False
    srcab: frozenset = frozenset()
    srcc: frozenset = frozenset()
    ws: int = 1
    succ: list = field(default_factory=list)


def _operands(rest: str) -> list[str]:
    # drop modifiers such as offset:16, and trailing comments
    rest = rest.split(";")[0]
    return [o.strip() for o in rest.split(",") if o.strip()]


def parse(lines: list[str]) -> list[Ins]:
    """Instructions of one kernel body, with control-flow successors."""
    ins: list[Ins] = []
    labels: dict[str, int] = {}
    for raw in lines:
        s = raw.strip()
        if not s or s.startswith((";", "//")):
            continue
        m = re.match(r"^([\w.$]+):", s)
        if m:
            labels[m.group(1)] = len(ins)
            continue
        if s.startswith("."):
            continue
        parts = s.split(None, 1)
        op = parts[0]
        ops = _operands(parts[1]) if len(parts) > 1 else []
        it = Ins(s, op)
        if op == "s_nop":
            it.ws = int(ops[0], 0) + 1 if ops else 1
        elif op.startswith("v_mfma"):
            it.mfma = True
            it.defs = _regs(ops[0])
            it.srcab = _regs(ops[1]) | _regs(ops[2])
            it.srcc = _regs(ops[3]) if len(ops) > 3 else frozenset()
            it.uses = it.srcab | it.srcc
        elif op.startswith(("ds_write", "ds_store", "global_store", "buffer_store", "flat_store")):
            it.uses = frozenset().union(*(_regs(o) for o in ops)) if ops else frozenset()
        elif op.startswith(("v_", "ds_", "global_", "buffer_", "flat_")):
            first = _regs(ops[0]) if ops else frozenset()
            lds_dma = op.startswith(("global_load_lds", "buffer_load")) and "lds" in s
            if op.startswith("v_cmp") or op.startswith(("v_readfirstlane", "v_readlane")) or lds_dma:
                it.uses = frozenset().union(*(_regs(o) for o in ops)) if ops else frozenset()
            else:
                it.defs = first
                it.uses = frozenset().union(*(_regs(o) for o in ops[1:])) if len(ops) > 1 else frozenset()
        ins.append(it)
    for i, it in enumerate(ins):
        if it.op == "s_endpgm":
            continue
        target = None
        if it.op.startswith(("s_branch", "s_cbranch")):
            ops = _operands(it.text.split(None, 1)[1])
            target = labels.get(ops[0]) if ops else None
        if it.op == "s_branch":
            it.succ = [target] if target is not None else []
        else:
            it.succ = ([i + 1] if i + 1 < len(ins) else []) + ([target] if target is not None else [])
    return ins


def _forward(ins: list[Ins], start: int, budget: int):
    """Instructions reachable after `start` within `budget` wait states."""
    seen = {}
    stack = [(s, 0) for s in ins[start].succ]
    while stack:
        j, w = stack.pop()
        if w >= budget or seen.get(j, budget + 1) <= w:
            continue
        seen[j] = w
        yield j
        for s in ins[j].succ:
            stack.append((s, w + ins[j].ws))


def check(ins: list[Ins]) -> list[str]:
    """Hazard descriptions (empty when every rule holds on every path)."""
    out = []
    preds: dict[int, list[int]] = {}
    for i, it in enumerate(ins):
        for s in it.succ:
            preds.setdefault(s, []).append(i)
    for i, it in enumerate(ins):
        if not it.mfma:
            continue
        # VALU (or any non-MFMA) write shortly before this MFMA reads it
        stack = [(p, 0) for p in preds.get(i, [])]
        seen = set()
        while stack:
            j, w = stack.pop()
            if w >= VALU_MFMA or j in seen:
                continue
            seen.add(j)
            pj = ins[j]
            if not pj.mfma and pj.defs & it.uses:
                out.append(f"VALU write -> MFMA read within {VALU_MFMA}: {pj.text} -> {it.text}")
            stack.extend((p, w + pj.ws) for p in preds.get(j, []))
        read_ws, war_ws = _waits(it.op)
        for j in _forward(ins, i, read_ws):
            nj = ins[j]
            if nj.mfma:
                if nj.srcab & it.defs:
                    out.append(f"MFMA write -> MFMA A/B read within {read_ws}: {it.text} -> {nj.text}")
                if nj.srcc & it.defs and nj.srcc != it.defs:
                    out.append(f"MFMA write -> partial C read within {read_ws}: {it.text} -> {nj.text}")
                continue
            if (nj.uses | nj.defs) & it.defs:
                out.append(f"MFMA write -> access within {read_ws}: {it.text} -> {nj.text}")
        if it.srcc and it.srcc != it.defs:
            for j in _forward(ins, i, war_ws):
                nj = ins[j]
                if not nj.mfma and nj.defs & it.srcc:
                    out.append(f"MFMA C read -> write within {war_ws}: {it.text} -> {nj.text}")
    return out


def kernels(asm_text: str) -> dict[str, list[str]]:
    """Kernel name -> body lines, from a device assembly file (functions named
    by `.type NAME,@function`)."""
    names = set(re.findall(r"^\s*\.type\s+([\w.$]+),\s*@function", asm_text, re.M))
    out: dict[str, list[str]] = {}
    name = None
    for line in asm_text.splitlines():
        m = re.match(r"^([\w.$]+):", line)
        if m and m.group(1) in names:
            name = m.group(1)
            out[name] = []
            continue
        if name is not None:
            # a kernel may hold several s_endpgm (early exits); its body ends
            # at the function's end label
            if line.strip().startswith(".Lfunc_end"):
                name = None
                continue
            out[name].append(line)
    return out
