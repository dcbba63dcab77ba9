"""Static check of gfx950 assembly: no instruction may touch the destination
registers of an LDS read that can still be in flight.

The hardware writes an LDS read's destination when the read returns, not when
it issues; LDS operations (reads, writes, cross-lane permutes) return in
issue order and all count against lgkmcnt, so `s_waitcnt lgkmcnt(N)`
guarantees that every LDS operation but the newest N has returned.  Reads the
compiler emits get their waits from the compiler; reads issued from inline
asm (or waits placed by hand) do not, and a register reused too early gives
wrong data or, as once happened with an epilogue address, a memory fault.

The check is a dataflow analysis over the kernel's control-flow graph.  The
state at a point is the set of LDS reads that may be in flight, each with the
smallest number of LDS operations issued after it along any path; at a join
the sets are merged (union, minimum), so a read is only taken as returned
when every path to the point has retired it.  Scalar loads share lgkmcnt but
only make reads retire earlier, so ignoring them is conservative.
"""
import re

_BRANCH = re.compile(r"^s_(c?branch\w*)\s+(\.LBB\w+)")


def _regs(tok):
    """Registers named by an operand: ('v', n) and ('a', n) keys."""
    m = re.match(r"([va])\[(\d+):(\d+)\]$", tok)
    if m:
        return [(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)]
    m = re.match(r"([va])(\d+)$", tok)
    return [(m.group(1), int(m.group(2)))] if m else []


def _returns_data(op):
    return op.startswith(("ds_read", "ds_bpermute", "ds_permute", "ds_swizzle", "ds_append", "ds_consume")) \
        or "_rtn" in op


def _instr(line):
    s = line.split(";")[0].strip()
    if not s or s.startswith(".") or s.endswith(":"):
        return None
    return s


def kernel_bodies(asm_text):
    """Map kernel symbol -> list of lines, from its label to the end of the
    function (blocks placed after s_endpgm included)."""
    out = {}
    lines = asm_text.split("\n")
    for i, l in enumerate(lines):
        m = re.match(r"^(_Z\S+):", l)
        if m and not l.startswith("\t"):
            body = []
            for x in lines[i + 1:]:
                if x.startswith(".Lfunc_end"):
                    break
                body.append(x)
            out[m.group(1)] = body
    return out


def _blocks(body):
    """Basic blocks: list of (label or None, [instructions], successors)."""
    blocks = []
    cur_label, cur = None, []

    def close():
        blocks.append([cur_label, list(cur), None])

    for l in body:
        m = re.match(r"^(\.LBB\w+):", l)
        if m:
            if cur or cur_label is not None:
                close()
            cur_label, cur = m.group(1), []
            continue
        s = _instr(l)
        if s is None:
            continue
        cur.append(s)
        op = s.split()[0]
        if op.startswith("s_branch") or op.startswith("s_cbranch") or op in ("s_endpgm", "s_setpc_b64"):
            close()
            cur_label, cur = None, []
    if cur or cur_label is not None:
        close()
    index = {b[0]: k for k, b in enumerate(blocks) if b[0]}
    for k, b in enumerate(blocks):
        succ = []
        last = b[1][-1] if b[1] else ""
        op = last.split()[0] if last else ""
        m = _BRANCH.match(last)
        if m:
            succ.append(index[m.group(2)])
        if op not in ("s_branch", "s_endpgm", "s_setpc_b64") and k + 1 < len(blocks):
            succ.append(k + 1)           # fall through (also after a conditional branch)
        b[2] = succ
    return blocks


def _step(state, s, where, bad):
    """Apply one instruction to state {read id: (regs, newer)}; record hazards."""
    op = s.split()[0]
    ops = [t.strip(",") for t in s.split()[1:]]
    if op == "s_waitcnt" and "lgkmcnt" in s:
        n = int(re.search(r"lgkmcnt\((\d+)\)", s).group(1))
        return {k: v for k, v in state.items() if v[1] < n}
    pending = {}
    for k, (regs, _) in state.items():
        for r in regs:
            pending[r] = k
    if op.startswith("ds_"):
        srcs = ops[1:] if _returns_data(op) else ops
        touched = [r for x in srcs for r in _regs(x) if r in pending]
        if touched:
            bad.append((where, s, touched[:4]))
        new = {k: (regs, newer + 1) for k, (regs, newer) in state.items()}
        if _returns_data(op):
            dst = set(_regs(ops[0]))
            # a newer read of the same registers lands after the older one (in order)
            new = {k: (regs - dst, newer) for k, (regs, newer) in new.items()}
            new = {k: v for k, v in new.items() if v[0]}
            new[where] = (frozenset(dst), 0)
        return new
    touched = [r for x in ops for r in _regs(x) if r in pending]
    if touched:
        bad.append((where, s, touched[:4]))
    return state


def _merge(a, b):
    out = dict(a)
    for k, (regs, newer) in b.items():
        if k in out:
            out[k] = (out[k][0] | regs, min(out[k][1], newer))
        else:
            out[k] = (regs, newer)
    return out


def hazards(body):
    """Violations in one kernel (empty list when clean): (instruction id,
    instruction, registers of an in-flight read it touches)."""
    blocks = _blocks(body)
    if not blocks:
        return []
    ins = {0: {}}
    work = [0]
    bad_all = {}
    while work:
        k = work.pop()
        state = ins[k]
        bad = []
        for j, s in enumerate(blocks[k][1]):
            state = _step(state, s, (k, j), bad)
        bad_all[k] = bad
        for t in blocks[k][2]:
            m = _merge(ins[t], state) if t in ins else dict(state)
            if t not in ins or m != ins[t]:
                ins[t] = m
                work.append(t)
    out = []
    for k in sorted(bad_all):
        out += [(w, s, [r[0] + str(r[1]) for r in t]) for w, s, t in bad_all[k]]
    return out
