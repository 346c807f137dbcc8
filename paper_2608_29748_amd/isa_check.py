"""Build-time check of the attention kernels' untracked LDS reads.

The bf16 attention kernel issues some LDS reads as inline assembly that the compiler's
wait insertion does not see (so that it does not also wait for the direct-to-LDS copies
of the next chunk), waits for them itself with ``s_waitcnt lgkmcnt(0)`` and only then
reads the registers.  That is sound only if the generated code leaves the destination
registers of such a read alone until the wait: the compiler takes the value as written
when the asm statement ends, so nothing stops it in principle from copying, spilling or
reusing those registers before the data arrive.  This module reads the gfx950 assembly
of a source and proves, by a data-flow pass over each kernel's control-flow graph, that
no instruction reads or writes a register such a read may still be writing.

LDS operations return in order, so after ``s_waitcnt lgkmcnt(N)`` at most the last N of
them are outstanding (scalar loads share the counter but only lower how many LDS
operations can remain).  The state at each point maps a pending register to the
smallest number of LDS operations issued after its read on any path there.
"""
from __future__ import annotations

import re
from typing import Dict, List, Tuple

_CAP = 64


def _vregs(tok: str) -> set:
    tok = tok.strip()
    m = re.match(r"v\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def _kernels(asm: str) -> Dict[str, List[Tuple[str, bool]]]:
    """Kernel name -> its lines as (instruction or label, inside an inline-asm block)."""
    out: Dict[str, List[Tuple[str, bool]]] = {}
    name = None
    inasm = False
    for raw in asm.split("\n"):
        ln = raw.strip()
        m = re.match(r"^([A-Za-z_][\w.$]*):", raw)
        if m and not raw.startswith((".L", "\t")) and name is None and m.group(1).startswith("_Z"):
            name = m.group(1)
            out[name] = []
            continue
        if name is None:
            continue
        if ln.startswith(".Lfunc_end"):
            name = None
            continue
        if ln.startswith(";;#ASMSTART"):
            inasm = True
            continue
        if ln.startswith(";;#ASMEND"):
            inasm = False
            continue
        code = ln.split(";")[0].strip()
        if code and (not code.startswith(".") or code.endswith(":")):
            out[name].append((code, inasm))
    return out


def _blocks(lines):
    """Basic blocks as (label, instructions, successor labels): a block starts at each
    label and after each branch or end of program."""
    raw = []   # (label, instructions)
    label, cur = "<entry>", []
    for code, inasm in lines:
        if code.endswith(":") and not inasm:
            raw.append((label, cur))
            label, cur = code[:-1], []
            continue
        cur.append((code, inasm))
        op = code.split()[0]
        if op == "s_branch" or op.startswith("s_cbranch") or op in ("s_endpgm", "s_setpc_b64"):
            raw.append((label, cur))
            label, cur = f"<after {len(raw)}>", []
    raw.append((label, cur))
    blocks = []
    for i, (lbl, ins) in enumerate(raw):
        nxt = [raw[i + 1][0]] if i + 1 < len(raw) else []
        last = ins[-1][0].split() if ins else [""]
        if last[0] == "s_branch":
            succ = [last[1]]
        elif last[0].startswith("s_cbranch"):
            succ = [last[1]] + nxt
        elif last[0] in ("s_endpgm", "s_setpc_b64"):
            succ = []
        else:
            succ = nxt
        blocks.append((lbl, ins, succ))
    return blocks


def _step(state: Dict[int, int], code: str, inasm: bool, bad: List[str]) -> Dict[int, int]:
    op, _, rest = code.partition(" ")
    operands = [x.strip() for x in re.split(r",\s*", rest)] if rest else []
    if op == "s_waitcnt":
        m = re.search(r"lgkmcnt\((\d+)\)", code)
        if m:
            n = int(m.group(1))
            state = {r: k for r, k in state.items() if k < n}
        return state
    if op.startswith("s_"):
        return state
    touched = set()
    for x in operands:
        touched |= _vregs(x)
    if op.startswith("ds_"):
        if inasm and op.startswith("ds_read"):
            dst = _vregs(operands[0]) if operands else set()
            if (touched - dst) & set(state):
                bad.append(code)
            state = {r: min(k + 1, _CAP) for r, k in state.items()}
            for r in dst:
                state[r] = 0
            return state
        if touched & set(state):
            bad.append(code)
        return {r: min(k + 1, _CAP) for r, k in state.items()}
    if touched & set(state):
        bad.append(code)
    return state


def check(asm: str) -> List[str]:
    """Violations ("kernel: instruction") over every kernel holding an inline-asm LDS read."""
    problems: List[str] = []
    for name, lines in _kernels(asm).items():
        if not any(inasm and code.startswith("ds_read") for code, inasm in lines):
            continue
        blocks = _blocks(lines)
        index = {b[0]: i for i, b in enumerate(blocks)}
        entry: List[Dict[int, int] | None] = [None] * len(blocks)
        entry[0] = {}
        work = [0]
        while work:
            i = work.pop()
            state = dict(entry[i])
            scratch: List[str] = []
            for code, inasm in blocks[i][1]:
                state = _step(state, code, inasm, scratch)
            for s in blocks[i][2]:
                j = index.get(s)
                if j is None:
                    continue
                old = entry[j]
                if old is None:
                    new = dict(state)
                else:
                    new = dict(old)
                    for r, k in state.items():
                        new[r] = min(k, new.get(r, _CAP))
                if new != old:
                    entry[j] = new
                    work.append(j)
        bad: List[str] = []
        for i, (_, ins, _) in enumerate(blocks):
            if entry[i] is None:
                continue
            state = dict(entry[i])
            for code, inasm in ins:
                state = _step(state, code, inasm, bad)
        problems += [f"{name}: {b}" for b in dict.fromkeys(bad)]
    return problems


def checked_kernels(asm: str) -> List[str]:
    return [n for n, lines in _kernels(asm).items()
            if any(inasm and code.startswith("ds_read") for code, inasm in lines)]
