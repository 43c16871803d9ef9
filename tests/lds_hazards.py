"""Static check of gfx950 assembly for registers of LDS reads still in flight.

Kernels that read LDS with inline-assembly ``ds_read_b128`` (so that the
compiler does not order the reads after LDS-direct loads of other ring
stages) must retire every such read with an explicit ``s_waitcnt
lgkmcnt`` before any instruction touches its destination registers: the
compiler does not know the read is pending, reuses the registers, and the
late LDS return then overwrites whatever they hold by then (an address,
say).  This module walks the control-flow graph of every kernel in an
assembly file and reports each instruction that, on some path, reads or
writes a VGPR of an LDS read that no ``s_waitcnt lgkmcnt`` has retired.

Model: LDS operations retire in order, ``lgkmcnt(N)`` keeps the N youngest
in flight; scalar memory loads share the counter but return out of order,
so while one is pending only ``lgkmcnt(0)`` retires anything.
"""
import re

_SMEM = frozenset({-1})


def _regs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return frozenset(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    if m:
        return frozenset({int(m.group(1))})
    return frozenset()


def _operands(line):
    parts = line.split(None, 1)
    if len(parts) < 2:
        return parts[0], []
    return parts[0], [o.strip() for o in re.split(r",(?![^\[]*\])", parts[1].split(";")[0])]


def _merge(a, b):
    n = max(len(a), len(b))
    a = (frozenset(),) * (n - len(a)) + a
    b = (frozenset(),) * (n - len(b)) + b
    return tuple(x | y for x, y in zip(a, b))


def _blocks(lines):
    blocks, cur = [], []
    for ln, raw in lines:
        s = raw.strip()
        m = re.match(r"^(\.LBB\S+|L\w+):", s)
        if m:
            if cur:
                blocks.append(cur)
            cur = [("label", m.group(1), ln)]
            continue
        if not s or s.startswith(";") or s.startswith("."):
            continue
        cur.append(("ins", s, ln))
        op = s.split()[0]
        if op.startswith("s_branch") or op.startswith("s_cbranch") or op == "s_endpgm" or op.startswith("s_setpc"):
            blocks.append(cur)
            cur = []
    if cur:
        blocks.append(cur)
    labels = {b[0][1]: i for i, b in enumerate(blocks) if b and b[0][0] == "label"}
    succ = []
    for i, b in enumerate(blocks):
        ins = [x for x in b if x[0] == "ins"]
        last = ins[-1][1] if ins else ""
        op = last.split()[0] if last else ""
        if op.startswith("s_branch"):
            s = [labels[last.split()[1]]]
        elif op.startswith("s_cbranch"):
            s = [labels[last.split()[1]], i + 1]
        elif op == "s_endpgm":
            s = []
        else:
            s = [i + 1]
        succ.append([x for x in s if x < len(blocks)])
    return blocks, succ


def hazards(lines):
    """lines: [(line_number, text)] of one kernel.  Returns {line: text} of
    the instructions that touch registers of an unretired LDS read."""
    blocks, succ = _blocks(lines)
    if not blocks:
        return {}
    state_in = [None] * len(blocks)
    state_in[0] = ()
    work, bad = [0], {}
    while work:
        i = work.pop()
        st = state_in[i]
        for kind, s, ln in blocks[i]:
            if kind != "ins":
                continue
            op, ops = _operands(s)
            if op == "s_waitcnt":
                m = re.search(r"lgkmcnt\((\d+)\)", s)
                if m:
                    n = int(m.group(1))
                    if n == 0:
                        st = ()
                    elif not any(-1 in p for p in st) and n < len(st):
                        st = st[len(st) - n:]
                continue
            is_read = op.startswith("ds_read") or op.startswith("ds_load")
            # an LDS read may target the registers of an older pending one
            # (they retire in order); its address must not be pending
            checked = ops[1:] if is_read else ops
            used = frozenset().union(*[_regs(o) for o in checked]) if checked else frozenset()
            if any(used & p for p in st):
                bad.setdefault(ln, s)
            if is_read:
                st = st + (_regs(ops[0]),)
            elif op.startswith("s_load") or op.startswith("s_buffer_load") or op.startswith("s_memtime"):
                st = st + (_SMEM,)
            elif op.startswith("ds_"):
                st = st + (frozenset(),)
            st = st[-32:]
        for j in succ[i]:
            new = st if state_in[j] is None else _merge(state_in[j], st)
            if new != state_in[j]:
                state_in[j] = new
                work.append(j)
    return bad


def kernels(asm_text):
    """Split an assembly file into {kernel symbol: [(line, text)]}."""
    out, cur = {}, None
    for i, line in enumerate(asm_text.splitlines()):
        m = re.match(r"^(_Z\S+):", line)
        if m and "kernel" in m.group(1):
            cur = m.group(1)
            out[cur] = []
            continue
        if cur is not None:
            if re.match(r"^\s*(\.section|\.Lfunc_end)", line):
                cur = None
                continue
            out[cur].append((i + 1, line))
    return out
