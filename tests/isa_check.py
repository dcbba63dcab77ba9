"""Static check of gfx950 assembly for in-flight inline-asm LDS reads.

The GEMM issues its fragment reads (ds_read_b128) through inline asm and
places the matching s_waitcnt lgkmcnt by hand.  The compiler treats an asm
output as written when the asm executes, but the hardware writes it when the
read returns; so from a read's issue until an s_waitcnt retires it, no other
instruction may touch its destination registers (reads retire in order).
This walks a kernel's instruction stream -- prologue, three iterations of its
main loop, and the loop exit up to the first lgkmcnt(0) -- and reports every
violation.
"""
import re


def _regs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return list(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return [int(m.group(1))] if m else []


def _returns_data(op):
    return op.startswith(("ds_read", "ds_bpermute", "ds_permute", "ds_swizzle", "ds_append", "ds_consume")) \
        or "_rtn" in op


def _instrs(lines):
    for l in lines:
        s = l.strip()
        if s and not s.startswith(";") and not s.endswith(":") and not s.startswith("."):
            yield s


class _Sim:
    """LDS operations (reads, writes, cross-lane permutes) retire in issue
    order and all count against lgkmcnt: lgkmcnt(N) guarantees every LDS op but the newest N has
    retired (scalar loads share the counter but only make more retire, so
    ignoring them is conservative).  Destination registers of unretired
    reads are the ones nothing else may touch."""

    def __init__(self):
        self.seq = 0
        self.queue = []        # issue sequence numbers of unretired LDS ops
        self.pending = {}      # register -> sequence number of its read

    def step(self, s):
        op = s.split()[0]
        ops = [t.strip(",") for t in s.split()[1:]]
        if op == "s_waitcnt" and "lgkmcnt" in s:
            n = int(re.search(r"lgkmcnt\((\d+)\)", s).group(1))
            self.queue = self.queue[-n:] if n else []
            live = set(self.queue)
            self.pending = {r: k for r, k in self.pending.items() if k in live}
            return None
        if op.startswith("ds_"):
            # every LDS instruction counts against lgkmcnt (cross-lane ds_bpermute
            # and friends included); those that return data write their first operand
            touched = [r for x in ops[1:] for r in _regs(x) if r in self.pending]
            self.seq += 1
            self.queue.append(self.seq)
            if _returns_data(op):
                for r in _regs(ops[0]):
                    self.pending[r] = self.seq
            else:
                touched += [r for r in _regs(ops[0]) if r in self.pending]
            return touched or None
        touched = [r for x in ops for r in _regs(x) if r in self.pending]
        return touched or None


def kernel_bodies(asm_text):
    """Map kernel symbol -> list of lines (from its label to s_endpgm)."""
    out = {}
    lines = asm_text.split("\n")
    for i, l in enumerate(lines):
        m = re.match(r"^(_Z\S+):", l)
        if m and not l.startswith("\t"):
            body = []
            for x in lines[i + 1:]:
                body.append(x)
                if "s_endpgm" in x:
                    break
            out[m.group(1)] = body
    return out


def hazards(body):
    """Violations in one kernel (empty list when clean)."""
    heads = [i for i, l in enumerate(body) if "Loop Header" in l]
    sim = _Sim()
    bad = []
    if not heads:
        for s in _instrs(body):
            t = sim.step(s)
            if t:
                bad.append(("body", s, t[:4]))
        return bad
    start = heads[0]
    end = next(i for i in range(start, len(body)) if re.search(r"s_cbranch_scc[01] \.LBB", body[i]))
    for s in _instrs(body[:start]):
        t = sim.step(s)
        if t:
            bad.append(("prologue", s, t[:4]))
    for it in range(3):
        for s in _instrs(body[start:end + 1]):
            t = sim.step(s)
            if t:
                bad.append(("iter%d" % it, s, t[:4]))
    for s in _instrs(body[end + 1:]):
        if s.startswith("s_waitcnt") and "lgkmcnt(0)" in s:
            break
        t = sim.step(s)
        if t:
            bad.append(("exit", s, t[:4]))
    return bad
