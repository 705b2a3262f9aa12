"""Static check of the gfx950 assembly for LDS reads written as inline asm.

The GEMM and attention kernels issue some LDS reads (ds_read_b128,
ds_read_b64_tr_b16) as inline asm and wait for them with their own
`s_waitcnt lgkmcnt(N)`, so that the reads of the next stage overlap the
MFMAs of this one. The compiler does not know that such a read's destination
registers are filled only later: if it places a copy, a bit-field merge or
any other use of those registers between the read and its wait, the kernel
reads stale values, and if it writes them there, the LDS return overwrites
the write. Nothing at run time reports either; the result is just wrong.

This module walks each kernel's control-flow graph and tracks, per program
point, the LDS operations still in flight, oldest first, with the VGPRs that
the inline-asm reads among them will write. LDS operations complete in issue
order, so `s_waitcnt lgkmcnt(N)` leaves at most the N newest in flight
(scalar-memory loads share the counter but may complete in any order, so
they are assumed to complete at once, which can only keep more LDS reads in
flight). Where paths join, the in-flight lists are aligned at their newest
entry and united. Any instruction that reads or writes a VGPR of an
in-flight inline-asm read is reported.
"""
import re
from collections import deque

_LABEL = re.compile(r"^(\.L[\w$.]+|[A-Za-z_][\w$.]*):")
_VRANGE = re.compile(r"^v\[(\d+):(\d+)\]")
_VONE = re.compile(r"^v(\d+)$")
_CAP = 32   # longest in-flight list kept; older entries are merged (sound)


def vgprs(tok):
    tok = tok.strip().split()[0] if tok.strip() else ""
    m = _VRANGE.match(tok)
    if m:
        return frozenset(range(int(m.group(1)), int(m.group(2)) + 1))
    m = _VONE.match(tok)
    return frozenset((int(m.group(1)),)) if m else frozenset()


class Instr:
    __slots__ = ("line", "text", "op", "asm", "srcs", "dsts", "lgkm", "kind", "target")

    def __init__(self, line, text, asm):
        self.line, self.text, self.asm = line, text, asm
        self.op = text.split()[0]
        ops = [x for x in text[len(self.op):].split(",")]
        regs = [vgprs(x) for x in ops]
        op = self.op
        self.kind = "other"
        self.target = None
        self.lgkm = None
        if op.startswith("s_waitcnt"):
            m = re.search(r"lgkmcnt\((\d+)\)", text)
            self.lgkm = int(m.group(1)) if m else None
            self.kind = "wait"
        elif op == "s_branch":
            self.kind, self.target = "jump", ops[0].strip()
        elif op.startswith("s_cbranch"):
            self.kind, self.target = "cjump", ops[0].strip()
        elif op in ("s_endpgm", "s_setpc_b64", "s_trap"):
            self.kind = "end"
        elif op.startswith("ds_"):
            self.kind = "lds"
        # which operands are read and which written
        stores = ("buffer_store", "global_store", "flat_store", "scratch_store", "ds_write")
        if op.startswith("s_"):
            self.srcs, self.dsts = frozenset(), frozenset()
        elif op.startswith(stores) or (op.startswith("buffer_load") and " lds" in text):
            self.srcs, self.dsts = frozenset().union(*regs), frozenset()
        else:
            self.dsts = regs[0] if regs else frozenset()
            self.srcs = frozenset().union(*regs[1:]) if len(regs) > 1 else frozenset()


def _functions(lines, name_re):
    """(name, [(line number, text, inside inline asm)]) of each matching kernel."""
    pat = re.compile(name_re)
    out, cur, body, in_asm = [], None, [], False
    for k, raw in enumerate(lines, 1):
        t = raw.strip()
        if cur is None:
            m = re.match(r"^(_Z\S*):", raw)
            if m and pat.search(m.group(1)):
                cur, body = m.group(1), []
            continue
        if re.match(r"^\.Lfunc_end\d+:", t):
            out.append((cur, body))
            cur = None
            continue
        if t.startswith(";;#ASMSTART"):
            in_asm = True
        elif t.startswith(";;#ASMEND"):
            in_asm = False
        elif t and not t.startswith((";", ".cfi")) and (not t.startswith(".") or _LABEL.match(t)):
            body.append((k, t.split(";")[0].strip(), in_asm))
    return out


def _blocks(body):
    """Basic blocks: (label or None, [Instr]) and successor lists."""
    blocks, labels = [], {}
    cur = None
    for k, t, asm in body:
        m = _LABEL.match(t)
        if m:
            cur = [m.group(1), []]
            labels[m.group(1)] = len(blocks)
            blocks.append(cur)
            continue
        if cur is None:
            cur = [None, []]
            blocks.append(cur)
        ins = Instr(k, t, asm)
        cur[1].append(ins)
        if ins.kind in ("jump", "cjump", "end"):
            cur = None
    succ = []
    for i, (_, ins) in enumerate(blocks):
        last = ins[-1] if ins else None
        s = []
        if last is not None and last.kind in ("jump", "cjump"):
            assert last.target in labels, f"unknown branch target {last.target}"
            s.append(labels[last.target])
        if (last is None or last.kind not in ("jump", "end")) and i + 1 < len(blocks):
            s.append(i + 1)
        succ.append(s)
    return blocks, succ


def _merge(a, b):
    n = max(len(a), len(b))
    pa = (frozenset(),) * (n - len(a)) + a
    pb = (frozenset(),) * (n - len(b)) + b
    return tuple(x | y for x, y in zip(pa, pb))


def _cap(state):
    if len(state) <= _CAP:
        return state
    extra = len(state) - _CAP
    return (frozenset().union(*state[:extra + 1]),) + state[extra + 1:]


def _step(state, ins, report=None):
    if ins.kind == "wait":
        if ins.lgkm is not None:
            state = state[len(state) - ins.lgkm:] if ins.lgkm < len(state) else state
            if ins.lgkm == 0:
                state = ()
        return state
    if report is not None:
        live = frozenset().union(*state) if state else frozenset()
        if ins.srcs & live:
            report.append((ins.line, "reads", sorted(ins.srcs & live), ins.text))
        elif ins.dsts & live and ins.kind != "lds":     # LDS returns in order
            report.append((ins.line, "writes", sorted(ins.dsts & live), ins.text))
    if ins.kind == "lds":
        is_read = ins.op.startswith("ds_read")
        state = _cap(state + ((ins.dsts if ins.asm and is_read else frozenset()),))
    return state


def check_function(body):
    """Hazards of one kernel: [(line, 'reads'|'writes', vgprs, instruction)]."""
    blocks, succ = _blocks(body)
    if not blocks:
        return []
    into = [None] * len(blocks)
    into[0] = ()
    work = deque([0])
    queued = {0}
    while work:
        i = work.popleft()
        queued.discard(i)
        st = into[i]
        for ins in blocks[i][1]:
            st = _step(st, ins)
        for j in succ[i]:
            new = st if into[j] is None else _merge(into[j], st)
            if new != into[j]:
                into[j] = new
                if j not in queued:
                    work.append(j)
                    queued.add(j)
    report = []
    for i, (_, ins) in enumerate(blocks):
        st = into[i]
        if st is None:
            continue            # unreachable block
        for x in ins:
            st = _step(st, x, report)
    return report


def check_asm(path, name_re=r"."):
    """{kernel name: hazards} for every kernel in the .s file whose mangled
    name matches name_re, and the number of inline-asm LDS reads seen."""
    with open(path) as f:
        lines = f.read().split("\n")
    result, n_reads = {}, 0
    for name, body in _functions(lines, name_re):
        n_reads += sum(1 for _, t, asm in body if asm and t.startswith("ds_read"))
        result[name] = check_function(body)
    return result, n_reads
