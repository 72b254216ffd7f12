"""Checks on the gfx950 assembly of the attention kernels (test infrastructure).

The direct HBM -> LDS loads are inline assembly, so the compiler's hazard
recognizer does not look at their operands.  On gfx9-family hardware a vector
memory instruction that reads an SGPR written by a VALU instruction (for
example ``v_readlane_b32`` reloading a spilled SGPR) needs five wait states in
between; without them it reads the old value.  ``dma_sgpr_hazards`` finds
every direct load whose SGPR operands (buffer descriptor, offset) were written
by a VALU instruction fewer than five wait states earlier, on every path into
the load: the walk back from a load continues through each branch that jumps
to a label it passes, as well as through the fall-through edge.
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


# VOP3b encodings: the second operand is an SGPR destination (carry or flag)
_SDST2 = re.compile(r"v_(add|sub|subrev|addc|subb|subbrev)_co_|v_div_scale_|v_mad_(u64_u32|i64_i32)")
_UNCOND = ("s_branch", "s_endpgm", "s_setpc_b64")


def _sgpr_writes(inst: str) -> set:
    """SGPRs (and M0, as -1) that a VALU instruction writes."""
    if not inst.startswith("v_") or " " not in inst:
        return set()
    ops = [o.strip() for o in inst.split(None, 1)[1].split(",")]
    dsts = ops[:2] if _SDST2.match(inst) else ops[:1]
    out = set()
    for d in dsts:
        out |= _sgprs(d)
        if d == "m0":
            out.add(-1)
    return out


def _entries(asm_text: str) -> list:
    """("label", name) and ("inst", text) entries of a listing, in order."""
    out = []
    for line in asm_text.splitlines():
        line = line.split(";")[0].strip()
        if not line or line.startswith("."):
            if line.startswith(".LBB") and line.endswith(":"):
                out.append(("label", line[:-1]))
            continue
        if line.endswith(":"):
            out.append(("label", line[:-1]))
            continue
        out.append(("inst", line))
    return out


def dma_sgpr_hazards_cfg(asm_text: str) -> list:
    """(writer, direct load, wait states) for every VALU write of an SGPR (or
    M0) that a direct load reads, fewer than five wait states before the load
    on some path through the function's branches."""
    ents = _entries(asm_text)
    branches = {}   # label -> indices of the branches that jump to it
    for i, (kind, text) in enumerate(ents):
        if kind == "inst" and text.startswith(("s_branch", "s_cbranch")):
            branches.setdefault(text.split()[-1], []).append(i)
    found = []
    for i, (kind, text) in enumerate(ents):
        if kind != "inst" or not is_direct_load(text):
            continue
        read = {-1}   # M0 holds the LDS address
        for tok in text.split(None, 1)[1].split(",")[1:]:
            read |= _sgprs(tok.split()[0] if tok.strip() else tok)
        seen = set()
        stack = [(i - 1, 0)]
        while stack:
            j, waits = stack.pop()
            while j >= 0 and waits < REQUIRED_WAIT_STATES:
                if (j, waits) in seen:
                    break
                seen.add((j, waits))
                kind_j, prev = ents[j]
                if kind_j == "label":
                    for b in branches.get(prev, []):
                        stack.append((b, waits))
                    if j > 0 and ents[j - 1][0] == "inst" and ents[j - 1][1].startswith(_UNCOND):
                        break   # no fall-through edge into this label
                    j -= 1
                    continue
                if prev.startswith("s_nop"):
                    parts = prev.split()
                    waits += (int(parts[1], 0) if len(parts) > 1 else 0) + 1
                    j -= 1
                    continue
                if _sgpr_writes(prev) & read:
                    found.append((prev, text, waits))
                waits += 1
                j -= 1
    return found


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
