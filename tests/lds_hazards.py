"""Static check of LDS/scalar-memory load results in gfx950 assembly.

A ds_read (or s_load) writes its destination registers when the data returns,
not when the instruction issues; until an `s_waitcnt lgkmcnt(n)` has retired
it, no instruction may read or write those registers.  The compiler enforces
this for loads it emits itself, but not for loads issued from inline assembly,
whose results it treats as available at once: if such a result is dead (or
copied) before the hand-placed wait, the register can be handed to other code
and the late write corrupts it.

check(asm_text) runs a forward dataflow over each function's control-flow
graph.  The state maps every lgkm-counted load that may be in flight to the
smallest number of younger lgkm-counted operations issued after it on any path
(its rank).  `lgkmcnt(n)` retires LDS loads of rank >= n (LDS returns in
order); scalar loads return out of order and retire only at lgkmcnt(0).  Any
instruction whose register operands meet the destination of an in-flight load
is reported.
"""
from __future__ import annotations

import re

_REG = re.compile(r"\b([vsa])(?:\[(\d+):(\d+)\]|(\d+)\b)")
_LABEL = re.compile(r"^([.\w$]+):")
_CNT = re.compile(r"lgkmcnt\((\d+)\)")
_RANK_CAP = 64


def regs(operands: str) -> frozenset:
    out = set()
    for m in _REG.finditer(operands):
        kind = m.group(1)
        if m.group(4) is not None:
            lo = hi = int(m.group(4))
        else:
            lo, hi = int(m.group(2)), int(m.group(3))
        out.update((kind, r) for r in range(lo, hi + 1))
    return frozenset(out)


def _functions(text: str):
    """Yields (name, [(line_no, line)]) for every function body: from a global
    label to the next `.Lfunc_end`, global label or the end of the text."""
    lines = text.splitlines()
    starts = [j for j, l in enumerate(lines) if re.match(r"^[A-Za-z_][\w$.]*:", l)]
    for k, start in enumerate(starts):
        name = lines[start].split(":")[0]
        stop = starts[k + 1] if k + 1 < len(starts) else len(lines)
        end = next((j for j in range(start, stop) if lines[j].startswith(".Lfunc_end")), stop)
        yield name, [(j + 1, lines[j]) for j in range(start + 1, end)]


def _parse(body):
    """Basic blocks: list of (label or None, [(line_no, mnemonic, operands)])."""
    blocks, cur = [], [None, []]
    for no, raw in body:
        line = raw.split(";")[0].rstrip()
        if not line.strip():
            continue
        m = _LABEL.match(line)
        if m:
            if cur[1] or cur[0] is not None:
                blocks.append(cur)
            cur = [m.group(1), []]
            continue
        s = line.strip()
        if s.startswith("."):
            continue
        parts = s.split(None, 1)
        mnem, ops = parts[0], (parts[1] if len(parts) > 1 else "")
        cur[1].append((no, mnem, ops))
        if mnem.startswith("s_cbranch") or mnem in ("s_branch", "s_endpgm", "s_setpc_b64"):
            blocks.append(cur)
            cur = [None, []]
    if cur[1] or cur[0] is not None:
        blocks.append(cur)
    return blocks


def _successors(blocks):
    index = {b[0]: k for k, b in enumerate(blocks) if b[0] is not None}
    succ = []
    for k, (_, insts) in enumerate(blocks):
        last = insts[-1] if insts else None
        nxt = [k + 1] if k + 1 < len(blocks) else []
        if last is None:
            succ.append(nxt)
        elif last[1] == "s_branch":
            succ.append([index[last[2].strip()]])
        elif last[1].startswith("s_cbranch"):
            succ.append(nxt + [index[last[2].strip()]])
        elif last[1] in ("s_endpgm", "s_setpc_b64"):
            succ.append([])
        else:
            succ.append(nxt)
    return succ


def _lgkm_load(mnem: str):
    """(counted, is_scalar, has_dest) of an instruction."""
    if mnem.startswith("ds_"):
        dest = any(t in mnem for t in ("read", "load", "_rtn", "swizzle", "permute", "bpermute"))
        return True, False, dest
    if mnem.startswith(("s_load", "s_buffer_load", "s_scratch_load")):
        return True, True, True
    return False, False, False


def _merge(a: dict, b: dict) -> dict:
    out = dict(a)
    for key, (rank, r, sc) in b.items():
        if key in out:
            out[key] = (min(out[key][0], rank), r, sc)
        else:
            out[key] = (rank, r, sc)
    return out


def _step(state: dict, inst, report):
    no, mnem, ops = inst
    used = regs(ops)
    for key, (rank, r, _) in state.items():
        hit = used & r
        if hit:
            report.append((no, mnem, ops, key, sorted(hit)))
    if mnem == "s_waitcnt" or mnem.startswith("s_waitcnt_lgkmcnt"):
        m = _CNT.search(ops)
        n = None
        if m:
            n = int(m.group(1))
        elif mnem.startswith("s_waitcnt_lgkmcnt"):
            n = int(ops.split(",")[-1].strip(), 0)
        if n is not None:
            state = {k: v for k, v in state.items()
                     if not ((v[2] and n == 0) or (not v[2] and v[0] >= n))}
        return state
    counted, scalar, dest = _lgkm_load(mnem)
    if counted:
        state = {k: (min(v[0] + 1, _RANK_CAP), v[1], v[2]) for k, v in state.items()}
        if dest:
            state[no] = (0, regs(ops.split(",")[0]), scalar)
    return state


def check_function(body) -> list:
    blocks = _parse(body)
    if not blocks:
        return []
    succ = _successors(blocks)
    ins = [None] * len(blocks)
    ins[0] = {}
    work = [0]
    while work:
        k = work.pop()
        state = dict(ins[k])
        for inst in blocks[k][1]:
            state = _step(state, inst, [])
        for s in succ[k]:
            new = state if ins[s] is None else _merge(ins[s], state)
            if new != ins[s]:
                ins[s] = new
                work.append(s)
    report = []
    for k, (_, insts) in enumerate(blocks):
        if ins[k] is None:
            continue
        state = dict(ins[k])
        for inst in insts:
            state = _step(state, inst, report)
    return report


def check(text: str, name_filter: str = "") -> dict:
    """{function: [(line, mnemonic, operands, load_line, registers)]} of the hazards found."""
    out = {}
    for name, body in _functions(text):
        if name_filter in name:
            out[name] = check_function(body)
    return out
