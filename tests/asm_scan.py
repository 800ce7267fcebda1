"""Checks on the generated gfx950 code of the decode kernels (test helper).

The compiler inserts the wait states between an MFMA and a VALU instruction that
reads its result or overwrites one of its operands only around instructions it
sees; an inline-asm block is opaque to it.  These checks walk back from every
inline-asm block in the device assembly:

  * WAR / WAW: no register the block writes may be referenced by an MFMA since the
    last compiler-visible write of that register (the asm would overwrite a register
    that the MFMA may still be reading, or whose MFMA result is still to come);
  * RAW: no register the block reads may have been written last by an MFMA;
  * DPP: a block whose first instruction reads a DPP operand starts with s_nop 4 or
    more (an EXEC write needs 5 wait states before a DPP read).

Block boundaries (labels) are walked through, which is conservative.
"""
from __future__ import annotations

import re

WINDOW = 40  # instructions walked back from each block


def _regs(text: str) -> set[int]:
    r = {int(x) for x in re.findall(r"\bv(\d+)\b", text)}
    for a, b in re.findall(r"v\[(\d+):(\d+)\]", text):
        r |= set(range(int(a), int(b) + 1))
    return r


def _operands(inst: str) -> list[str]:
    parts = inst.split(None, 1)
    if len(parts) < 2:
        return []
    ops = parts[1].split(";")[0]
    return [o.strip() for o in re.split(r",(?![^\[]*\])", ops)]


def _dst(inst: str) -> set[int]:
    ops = _operands(inst)
    return _regs(ops[0]) if ops else set()


def _src(inst: str) -> set[int]:
    r: set[int] = set()
    for o in _operands(inst)[1:]:
        r |= _regs(o)
    return r


def _instructions(lines: list[str], start: int, step: int):
    k = start
    while 0 <= k < len(lines):
        t = lines[k].strip()
        k += step
        if not t or t.startswith(";") or t.startswith(".") or t.startswith("s_nop"):
            continue
        if re.match(r"^_Z\S*:", t):
            return
        yield t


def scan(asm_text: str) -> dict:
    """Returns {'blocks': n, 'war': [...], 'raw': [...], 'dpp': [...]}."""
    lines = asm_text.split("\n")
    out = {"blocks": 0, "war": [], "raw": [], "dpp": []}
    i = 0
    while i < len(lines):
        if ";;#ASMSTART" not in lines[i]:
            i += 1
            continue
        j = i
        while ";;#ASMEND" not in lines[j]:
            j += 1
        raw_body = [x.strip() for x in lines[i + 1:j] if x.strip() and not x.strip().startswith(";")]
        body = [x for x in raw_body if not x.startswith("s_nop")]
        if body:
            out["blocks"] += 1
            if "_dpp" in body[0].split()[0]:
                first = raw_body[0]
                if not (first.startswith("s_nop") and int(first.split()[1]) >= 4):
                    out["dpp"].append(body[0])
            writes: set[int] = set()
            reads: set[int] = set()
            for x in body:
                writes |= _dst(x)
                reads |= _src(x)
            pend_w, pend_r = set(writes), set(reads)
            for n, x in enumerate(_instructions(lines, i - 1, -1)):
                if n >= WINDOW or not (pend_w or pend_r):
                    break
                d = _dst(x)
                if x.startswith("v_mfma"):
                    hit = _regs(x) & pend_w
                    if hit:
                        out["war"].append((body[0], x, sorted(hit)))
                        pend_w -= hit
                    hit = d & pend_r
                    if hit:
                        out["raw"].append((body[0], x, sorted(hit)))
                        pend_r -= hit
                else:
                    pend_w -= d
                    pend_r -= d
        i = j + 1
    return out
