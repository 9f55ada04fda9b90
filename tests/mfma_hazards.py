"""Dependency-distance check of inline-assembly MFMAs in gfx950 device assembly.

The compiler inserts the wait states the matrix cores need between its own
MFMA instructions and their neighbours, but it treats an MFMA written as
inline assembly as an opaque statement: plain VALU code may be scheduled
right next to it, and registers it still reads may be reused.  This module
scans a kernel's assembly (``hipcc --cuda-device-only -S``) for three
patterns, counting one wait state per instruction and N+1 for ``s_nop N``:

* ``A``: a VALU instruction (``v_accvgpr_write`` included) writes a register
  that a following MFMA reads as A, B or C operand with fewer than 2 wait
  states between them;
* ``B``: an MFMA writes a register that a following non-MFMA instruction
  (VALU, LDS or memory) reads or writes with fewer than 11 wait states
  between them (an 8-pass MFMA; an MFMA issued in between counts as 8, since
  it cannot issue before the previous one has finished its passes);
* ``C``: an MFMA reads a register as C operand and a following VALU
  instruction writes it with fewer than 7 wait states between them (the
  accumulator input is read during the passes, not at issue).

Sequences are followed backwards through labels into every predecessor (the
fall-through block and every branch to the label), so dependencies across
branch edges and loop back-edges are covered.
"""
from __future__ import annotations

import re
from dataclasses import dataclass

VALU_TO_MFMA = 2
MFMA_TO_OTHER = 11
MFMA_SRCC_WAR = 7
MFMA_AS_WAIT = 8


@dataclass(frozen=True)
class Hazard:
    kind: str
    first: str
    second: str
    wait_states: int


def _regs(op: str) -> set:
    op = op.strip()
    m = re.match(r"^([va])\[(\d+):(\d+)\]$", op)
    if m:
        return {(m.group(1), k) for k in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"^-?\|?([va])(\d+)\|?$", op)
    if m:
        return {(m.group(1), int(m.group(2)))}
    return set()


def _union(ops) -> set:
    out = set()
    for o in ops:
        out |= _regs(o)
    return out


def _parse(text: str):
    """(kind, detail, written registers, read registers) of one line."""
    if re.match(r"^\.LBB\d+_\d+:", text):
        return ("label", text.split(":")[0], set(), set())
    parts = text.split(None, 1)
    op = parts[0]
    ops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
    if op.startswith("v_mfma"):
        return ("mfma", op, _regs(ops[0]), (_regs(ops[1]) | _regs(ops[2]), _regs(ops[3])))
    if op == "s_nop":
        return ("nop", int(ops[0], 0) + 1, set(), set())
    if op.startswith("v_"):
        if not ops:
            return ("valu", op, set(), set())
        if op.startswith("v_cmp") and not op.startswith("v_cmpx"):
            return ("valu", op, set(), _union(ops[1:]))
        return ("valu", op, _regs(ops[0]), _union(ops[1:]))
    if op.startswith(("ds_", "global_", "buffer_", "scratch_", "flat_")):
        if op.startswith(("ds_read", "ds_bpermute", "ds_permute", "global_load", "buffer_load",
                          "scratch_load", "flat_load")):
            return ("mem", op, _regs(ops[0]) if ops else set(), _union(ops[1:]))
        return ("mem", op, set(), _union(ops))
    if op == "s_branch" or op.startswith("s_cbranch"):
        return ("branch", ops[0] if ops else "", set(), set())
    if op == "s_endpgm":
        return ("end", op, set(), set())
    return ("other", op, set(), set())


def kernel_lines(asm: str, kernel: str) -> list:
    lines = asm.split("\n")
    start = next(i for i, l in enumerate(lines) if l.startswith(kernel + ":"))
    end = next(i for i in range(start, len(lines)) if lines[i].startswith(".Lfunc_end"))
    out = []
    for l in lines[start + 1:end]:
        t = l.split(";")[0].strip()
        if not t:
            continue
        if t.startswith(".") and not re.match(r"^\.LBB\d+_\d+:", t):
            continue
        out.append(t)
    return out


def scan_lines(lines: list) -> list:
    P = [(t, _parse(t)) for t in lines]
    labels = {p[1]: k for k, (_, p) in enumerate(P) if p[0] == "label"}
    preds: dict = {}
    for k, (t, p) in enumerate(P):
        if p[0] == "branch" and p[1] in labels:
            preds.setdefault(p[1], []).append(k)
        if p[0] == "label" and k > 0:
            prev_t, prev = P[k - 1]
            if not (prev[0] == "branch" and prev_t.startswith("s_branch")) and prev[0] != "end":
                preds.setdefault(p[1], []).append(k - 1)

    def back(k, depth, seen):
        seq = []
        j = k
        while j >= 0 and len(seq) < depth:
            p = P[j][1]
            if p[0] == "label":
                out = []
                for q in preds.get(p[1], []):
                    key = (p[1], q, len(seq))
                    if key in seen:
                        continue
                    seen.add(key)
                    for tail in back(q, depth - len(seq), seen):
                        out.append(seq + tail)
                return out or [seq]
            seq.append(j)
            j -= 1
        return [seq]

    def cost(j, mfma_cost):
        p = P[j][1]
        if p[0] == "mfma":
            return mfma_cost
        if p[0] == "nop":
            return p[1]
        return 0 if p[0] == "label" else 1

    found = set()
    for k, (t, p) in enumerate(P):
        if p[0] not in ("mfma", "valu", "mem"):
            continue
        for seq in back(k - 1, 48, set()):
            w = wb = 0
            for j in seq:
                tj, pj = P[j]
                if p[0] == "mfma" and pj[0] == "valu":
                    if pj[2] & (p[3][0] | p[3][1]) and w < VALU_TO_MFMA:
                        found.add(Hazard("A", tj, t, w))
                if pj[0] == "mfma" and p[0] in ("valu", "mem"):
                    if pj[2] & (p[3] | p[2]) and wb < MFMA_TO_OTHER:
                        found.add(Hazard("B", tj, t, wb))
                    if p[0] == "valu" and pj[3][1] & p[2] and not pj[2] & p[2] and w < MFMA_SRCC_WAR:
                        found.add(Hazard("C", tj, t, w))
                w += cost(j, 1)
                wb += cost(j, MFMA_AS_WAIT)
                if w >= MFMA_TO_OTHER and wb >= MFMA_TO_OTHER:
                    break
    return sorted(found, key=lambda h: (h.kind, h.first, h.second))


def scan(asm: str, kernel: str) -> list:
    return scan_lines(kernel_lines(asm, kernel))
