"""Checks on the gfx950 assembly of the attention kernels (test infrastructure).

The direct HBM -> LDS loads are inline assembly, so the compiler's hazard
recognizer does not look at their operands.  On gfx9-family hardware a vector
memory instruction that reads an SGPR written by a VALU instruction (for
example ``v_readlane_b32`` reloading a spilled SGPR) needs five wait states in
between; without them it reads the old value.  ``dma_sgpr_hazards`` finds
every direct load whose SGPR operands (buffer descriptor, offset) were written
by a VALU instruction fewer than five wait states earlier.
"""
from __future__ import annotations

import re

REQUIRED_WAIT_STATES = 5


def _sgprs(tok: str) -> set:
    tok = tok.strip()
    m = re.fullmatch(r"s\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.fullmatch(r"s(\d+)", tok)
    if m:
        return {int(m.group(1))}
    return set()


def instructions(asm_text: str) -> list:
    """Instruction lines of an assembly listing (labels, directives, comments dropped)."""
    out = []
    for line in asm_text.splitlines():
        line = line.split(";")[0].strip()
        if not line or line.startswith(".") or line.endswith(":"):
            continue
        out.append(line)
    return out


def is_direct_load(inst: str) -> bool:
    return inst.startswith("buffer_load") and inst.split()[-1] == "lds"


def dma_sgpr_hazards(insts: list) -> list:
    """(writer, direct load, wait states) for every unresolved VALU->SGPR->load pair."""
    found = []
    for i, inst in enumerate(insts):
        if not is_direct_load(inst):
            continue
        operands = inst.split(None, 1)[1].split(",")
        read = set()
        for tok in operands[1:]:
            read |= _sgprs(tok.split()[0] if tok.strip() else tok)
        waits = 0
        for j in range(i - 1, -1, -1):
            prev = insts[j]
            if waits >= REQUIRED_WAIT_STATES:
                break
            if prev.startswith("s_nop"):
                parts = prev.split()
                waits += (int(parts[1], 0) if len(parts) > 1 else 0) + 1
                continue
            if prev.startswith("v_") and " " in prev:
                dst = prev.split(None, 1)[1].split(",")[0]
                if _sgprs(dst) & read:
                    found.append((prev, inst, waits))
            waits += 1
    return found
