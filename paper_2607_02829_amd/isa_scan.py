"""Scan of gfx950 assembly for reads of registers that an LDS load is still filling.

The MFMA kernels issue their LDS fragment reads as inline assembly, so that the compiler does not
make them wait for global-to-LDS fills in flight; the compiler then does not know when those
registers are written.  The kernels wait (s_waitcnt lgkmcnt) before using them, which is only
sound if no instruction -- a copy, a spill, another use, or the kernel's own consumer -- touches a
destination register between the read and the wait that retires it.  This scan checks exactly
that on the compiled code: LDS reads retire in issue order, s_waitcnt lgkmcnt(N) leaves the last N
in flight, and any vector instruction reading or writing a register of a read still in flight is
reported.

The check follows the control flow: the function is split into basic blocks (labels, branches,
fall-through), and the reads in flight at a block's entry are the union over its predecessors,
aligned from the newest read (a wait that leaves N in flight then keeps at least what it keeps on
every path), iterated to a fixed point over loops.  A wait on code that is laid out between a
branch and its target therefore does not clear reads on the path that jumps over it."""
from __future__ import annotations

import re

_LABEL = re.compile(r"^(\.LBB\d+_\d+):")
_MAXLEN = 64   # bound of the tracked list (the hardware counter holds far fewer)


def _regs(tok: str) -> set:
    m = re.match(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"([va])(\d+)$", tok)
    if m:
        return {(m.group(1), int(m.group(2)))}
    return set()


def _blocks(body: list[str]):
    """[(label or None, [instruction lines])] in layout order; a block ends at a label or after a
    branch / end instruction."""
    blocks, cur, lab = [], [], None
    for line in body:
        t = line.strip()
        m = _LABEL.match(t)
        if m:
            if cur or lab is not None:
                blocks.append((lab, cur))
            lab, cur = m.group(1), []
            continue
        if not t or t.startswith(";") or t.startswith(".") or t.endswith(":"):
            continue
        cur.append(t)
        op = t.split()[0]
        if op.startswith("s_branch") or op.startswith("s_cbranch") or op in ("s_endpgm", "s_setpc_b64"):
            blocks.append((lab, cur))
            lab, cur = None, []
    if cur or lab is not None:
        blocks.append((lab, cur))
    return blocks


def _merge(a: list, b: list) -> list:
    """Union of two in-flight lists aligned from the newest entry."""
    n = max(len(a), len(b))
    out = []
    for k in range(n, 0, -1):   # k-th newest
        s = set()
        if k <= len(a):
            s |= a[-k]
        if k <= len(b):
            s |= b[-k]
        out.append(frozenset(s))
    return out[-_MAXLEN:]


def _run(block: list[str], pending: list, count: bool):
    """Pending list after the block, and (if count) the instructions touching in-flight registers."""
    pending = list(pending)
    hits = []
    for t in block:
        op = t.split()[0]
        if op == "s_waitcnt":
            m = re.search(r"lgkmcnt\((\d+)\)", t)
            if m:
                n = int(m.group(1))
                pending = pending[max(0, len(pending) - n):] if n else []
            continue
        ops = [x.strip(",") for x in t.split()[1:]]
        live = set().union(*pending) if pending else set()
        if op.startswith("ds_read") or op.startswith("ds_load"):
            srcs = set().union(*(_regs(x) for x in ops[1:])) if len(ops) > 1 else set()
            if count and srcs & live:
                hits.append(t)
            pending.append(frozenset(_regs(ops[0]) if ops else set()))
            pending = pending[-_MAXLEN:]
            continue
        if op.startswith("s_"):
            continue
        touched = set().union(*(_regs(x) for x in ops)) if ops else set()
        if count and touched & live:
            hits.append(t)
    return pending, hits


def kernel_findings(asm: str) -> dict:
    """{kernel symbol: [instructions touching registers of an LDS read in flight]}."""
    out = {}
    for name in re.findall(r"^(_Z\S+):", asm, re.M):
        a = re.search(r"^" + re.escape(name) + r":", asm, re.M).start()
        b = asm.find(".Lfunc_end", a)
        blocks = _blocks(asm[a:b].split("\n")[1:])
        index = {lab: i for i, (lab, _) in enumerate(blocks) if lab is not None}
        succ = []
        for i, (_, ins) in enumerate(blocks):
            last = ins[-1].split() if ins else [""]
            s = []
            if last[0].startswith("s_branch"):
                s = [index[last[1]]] if len(last) > 1 and last[1] in index else []
            elif last[0].startswith("s_cbranch"):
                if len(last) > 1 and last[1] in index:
                    s.append(index[last[1]])
                if i + 1 < len(blocks):
                    s.append(i + 1)
            elif last[0] in ("s_endpgm", "s_setpc_b64"):
                s = []
            elif i + 1 < len(blocks):
                s = [i + 1]
            succ.append(s)
        entry = [None] * len(blocks)
        entry[0] = []
        work = [0]
        while work:
            i = work.pop()
            after, _ = _run(blocks[i][1], entry[i], False)
            for j in succ[i]:
                new = after if entry[j] is None else _merge(entry[j], after)
                if entry[j] is None or new != entry[j]:
                    entry[j] = new
                    work.append(j)
        hits = []
        for i, (_, ins) in enumerate(blocks):
            if entry[i] is not None:
                hits += _run(ins, entry[i], True)[1]
        out[name] = hits
    return out


def kernel_hazards(asm: str) -> dict:
    """{kernel symbol: number of instructions touching registers of an LDS read in flight}."""
    return {k: len(v) for k, v in kernel_findings(asm).items()}
