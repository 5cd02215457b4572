"""Scan of gfx950 assembly for reads of registers that an LDS load is still filling.

The MFMA kernels issue their LDS fragment reads as inline assembly, so that the compiler does not
make them wait for global-to-LDS fills in flight; the compiler then does not know when those
registers are written.  The kernels wait (s_waitcnt lgkmcnt) before using them, which is only
sound if no instruction the compiler placed -- a copy, a spill, another use -- touches a
destination register between the read and the wait that retires it.  This scan checks exactly
that on the compiled code: LDS reads retire in issue order, s_waitcnt lgkmcnt(N) leaves the last N
in flight, and any vector instruction reading or writing a register of a read still in flight
is reported.  Branch targets are taken conservatively (tracking continues across labels)."""
from __future__ import annotations

import re


def _regs(tok: str) -> set:
    m = re.match(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"([va])(\d+)$", tok)
    if m:
        return {(m.group(1), int(m.group(2)))}
    return set()


def kernel_hazards(asm: str) -> dict:
    """{kernel symbol: number of instructions touching registers of an LDS read in flight}."""
    out = {}
    for name in re.findall(r"^(_Z\S+):", asm, re.M):
        a = asm.index(name + ":")
        b = asm.find(".Lfunc_end", a)
        pending: list = []   # register sets of the LDS reads in flight, oldest first
        hits = 0
        for line in asm[a:b].split("\n"):
            t = line.strip()
            if not t or t.startswith(";") or t.endswith(":") or t.startswith("."):
                continue
            op = t.split()[0]
            if op == "s_waitcnt":
                m = re.search(r"lgkmcnt\((\d+)\)", t)
                if m:
                    n = int(m.group(1))
                    pending = pending[len(pending) - n:] if n else []
                continue
            ops = [x.strip(",") for x in t.split()[1:]]
            live = set().union(*pending) if pending else set()
            if op.startswith("ds_read") or op.startswith("ds_load"):
                srcs = set().union(*(_regs(x) for x in ops[1:])) if len(ops) > 1 else set()
                if srcs & live:
                    hits += 1
                pending.append(_regs(ops[0]) if ops else set())
                continue
            if op.startswith("s_"):
                continue
            touched = set().union(*(_regs(x) for x in ops)) if ops else set()
            if touched & live:
                hits += 1
        out[name] = hits
    return out
