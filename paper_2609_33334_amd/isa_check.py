"""Build-time checks of the gfx950 assembly of kernels that issue loads from inline asm.

Some kernels issue global loads from inline asm so that the compiler does not track
them (its own waits would also drain the global->LDS copies in flight).  The compiler
then believes those registers are ready at once, so two properties must hold in the
generated code, and ``build()`` refuses to write the library when either fails:

1. Waits.  On every control-flow path from such a load (global_load_dword[x4] between
   ;;#ASMSTART and ;;#ASMEND) an ``s_waitcnt vmcnt(N)`` with at least N vector-memory
   operations issued since the load comes before any instruction that names one of the
   load's destination registers.  Paths are tracked as (instruction, operations since the
   load) states, so loops and branches are covered exactly.
2. No spills.  A kernel of such a file with a nonzero private segment keeps values in
   scratch memory; a register the compiler spills or copies may be an asm load's
   destination before its wait, so those kernels must not spill at all.
"""
from __future__ import annotations

import re
from collections import deque

VMEM = re.compile(r'^(global_|buffer_|flat_)')
REG = re.compile(r'\bv(\d+)\b|\bv\[(\d+):(\d+)\]')
LABEL = re.compile(r'^(\.LBB\w+|\.Ltmp\w*):')
ASM_LOAD = re.compile(r'global_load_dword(x4)?\s')
# source markers of kernels that issue untracked loads from asm
ASM_LOAD_USERS = ("async_load16(", "async_load4(", "dma16(", "dma16_sbase(")


def _regs(text):
    out = set()
    for m in REG.finditer(text):
        if m.group(1):
            out.add(int(m.group(1)))
        else:
            out.update(range(int(m.group(2)), int(m.group(3)) + 1))
    return out


def _parse(lines):
    """-> list of (instruction text, inside an asm block) and a label -> index map."""
    ins, labels, in_asm = [], {}, False
    for line in lines:
        s = line.strip()
        if ';;#ASMSTART' in s:
            in_asm = True
            continue
        if ';;#ASMEND' in s:
            in_asm = False
            continue
        m = LABEL.match(s)
        if m:
            labels[m.group(1)] = len(ins)
            continue
        t = s.split(';')[0].strip()
        if not t or t.startswith('.') or t.endswith(':'):
            continue
        ins.append((t, in_asm))
    return ins, labels


def _succ(ins, labels, i):
    t = ins[i][0]
    op = t.split()[0]
    if op == 's_endpgm' or op.startswith('s_setpc'):
        return []
    if op == 's_branch':
        return [labels[t.split()[1]]]
    if op.startswith('s_cbranch'):
        return [i + 1, labels[t.split()[1]]]
    return [i + 1]


def check_kernel(lines, name, report=None):
    """(asm loads found, loads touched before a covering wait) in one kernel's code."""
    ins, labels = _parse(lines)
    nload = bad = 0
    for i, (t, asm) in enumerate(ins):
        if not (asm and ASM_LOAD.match(t)):
            continue
        nload += 1
        dst = _regs(t.split()[1].rstrip(','))
        seen = set()
        q = deque((s, 0) for s in _succ(ins, labels, i))
        while q:
            j, cnt = q.popleft()
            if j >= len(ins) or (j, cnt) in seen:
                continue
            seen.add((j, cnt))
            u = ins[j][0]
            mw = re.match(r's_waitcnt\s+.*vmcnt\((\d+)\)', u)
            if mw and cnt >= int(mw.group(1)):
                continue                      # covered on this path
            ops = u.split(None, 1)
            if len(ops) > 1 and _regs(ops[1]) & dst:
                if report is not None:
                    report.append(f"{name}: asm load {t.split()[1]} read before its wait: {u}")
                bad += 1
                break
            c2 = min(cnt + (1 if VMEM.match(u) else 0), 64)
            for s in _succ(ins, labels, j):
                q.append((s, c2))
    return nload, bad


def scratch_sizes(text):
    """{kernel symbol: private segment bytes} from the kernel descriptors of an assembly file."""
    out, cur = {}, None
    for line in text.splitlines():
        s = line.strip()
        if s.startswith('.amdhsa_kernel '):
            cur = s.split()[1]
        elif cur is not None and s.startswith('.amdhsa_private_segment_fixed_size'):
            out[cur] = int(s.split()[1])
            cur = None
    return out


def check_asm(path, only=None, report=None):
    """(asm loads checked, wait violations, spilling kernels) over one assembly file.
    ``report`` (a list) collects one line per problem."""
    text = open(path).read()
    src = text.splitlines()
    starts = [i for i, l in enumerate(src) if re.match(r'^_Z\S+:', l)]
    tot = bad = 0
    for k, s0 in enumerate(starts):
        e = starts[k + 1] if k + 1 < len(starts) else len(src)
        name = src[s0].split(':')[0]
        if only and only not in name:
            continue
        n, b = check_kernel(src[s0:e], name[-60:], report)
        tot += n
        bad += b
    spills = 0
    for name, size in scratch_sizes(text).items():
        if only and only not in name:
            continue
        if size:
            spills += 1
            if report is not None:
                report.append(f"{name[-60:]}: private segment of {size} bytes (spills)")
    return tot, bad, spills


def uses_asm_loads(source_text: str) -> bool:
    return any(m in source_text for m in ASM_LOAD_USERS)
