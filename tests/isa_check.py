"""Check of the fused kernel's hand-counted memory waits on its own built ISA.

The fused top-1 kernel issues some vector loads as inline assembly (the
[Vt;Q_e] operands into registers, the W1 ring into LDS) and waits for them
with explicit vmcnt counts; the compiler does not see those loads.  If the
compiler ever touched a destination register of such a load before a wait
that covers it -- for instance by spilling it to scratch -- the kernel would
read data that has not arrived.  This module walks every control-flow path
of a kernel in the compiler's assembly output (hipcc -S, gfx950) from each
register-destination buffer load and reports any instruction that reads or
writes its registers before an s_waitcnt vmcnt(N) with N no larger than the
number of vector-memory operations issued after it (they complete in order;
scratch, store and atomic operations count too)."""
import re

_VMEM = re.compile(r"^(buffer|global|scratch|flat)_(load|store|atomic)")


def kernel_body(asm: str, name: str):
    """Instructions and label positions of one kernel in an assembly file."""
    i = asm.index(f"\n{name}:")
    j = asm.index(".Lfunc_end", i)
    insts, labels = [], {}
    for line in asm[i:j].splitlines()[1:]:
        s = line.split(";")[0].strip()
        if not s:
            continue
        m = re.match(r"^(\.LBB\w+):", s)
        if m:
            labels[m.group(1)] = len(insts)
            continue
        if s.startswith("."):
            continue
        insts.append(s)
    return insts, labels


def _regs(text: str):
    out = set()
    for m in re.finditer(r"\bv\[(\d+):(\d+)\]", text):
        out |= set(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"(?<![\w\[:])v(\d+)\b", text):
        out.add(int(m.group(1)))
    return out


def _succ(insts, labels, i):
    y = insts[i]
    op = y.split()[0]
    if op == "s_endpgm":
        return []
    m = re.search(r"s_c?branch\w*\s+(\.LBB\w+)", y)
    if m:
        t = labels[m.group(1)]
        return [t] if op == "s_branch" else [t, i + 1]
    return [i + 1]


def hazards(insts, labels, scratch=False):
    """(loads checked, list of hazard descriptions).  Every buffer load into
    registers is followed until a covering wait and must not have its
    registers touched first.  With scratch=True loads into LDS are followed
    too, and every scratch access (the compiler's spills) issued while a
    buffer load is outstanding is listed."""
    found, loads = [], 0
    for i, y in enumerate(insts):
        if not y.startswith("buffer_load") and not y.startswith("global_load_lds"):
            continue
        m = re.match(r"buffer_load_dwordx4 v\[(\d+):(\d+)\]", y)
        lds = " lds" in y or y.startswith("global_load_lds")
        if (lds and not scratch) or (not lds and not m):
            continue
        loads += 1
        R = set() if lds else set(range(int(m.group(1)), int(m.group(2)) + 1))
        seen = set()
        stack = [(j, 0) for j in _succ(insts, labels, i)]
        while stack:
            j, M = stack.pop()
            if (j, M) in seen or j >= len(insts):
                continue
            seen.add((j, M))
            z = insts[j]
            w = re.search(r"s_waitcnt\s.*vmcnt\((\d+)\)", z)
            if w and int(w.group(1)) <= M:
                continue
            if z.startswith("s_endpgm"):
                found.append(f"load {i} {y!r}: reaches s_endpgm without a covering wait")
                continue
            if scratch and z.startswith("scratch_"):
                found.append(f"load {i} {y!r}: scratch access at {j} {z!r} before its wait")
                continue
            if _VMEM.match(z):
                dst = _regs(z.split(",")[0]) if "_load" in z.split()[0] else set()
                if (_regs(z) & R) and not (dst & R and not (_regs(",".join(z.split(",")[1:])) & R)):
                    found.append(f"load {i} {y!r}: registers touched at {j} {z!r}")
                for s2 in _succ(insts, labels, j):
                    stack.append((s2, min(M + 1, 64)))
                continue
            if _regs(z) & R:
                found.append(f"load {i} {y!r}: registers touched at {j} {z!r}")
                continue
            for s2 in _succ(insts, labels, j):
                stack.append((s2, M))
    return loads, found
