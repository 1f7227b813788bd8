"""Control-flow-aware check of gfx950 assembly for the kernels' asm register loads.

The scoring kernels issue some global loads from inline asm so that the compiler does
not track them (its own waits would also drain the global->LDS copies in flight).  The
compiler then believes those registers are ready at once.  This checker walks every
control-flow path from each such load (global_load_dword[x4] between ;;#ASMSTART and
;;#ASMEND) and requires an s_waitcnt vmcnt(N) with at least N vector-memory operations
issued since the load before any instruction mentions the load's destination registers.
Paths are tracked as (instruction, operations-since-load) states, so loops and the
dummy/real copy selects are covered exactly."""
import re, sys
from collections import deque

VMEM = re.compile(r'^(global_|buffer_|flat_)')
REG = re.compile(r'\bv(\d+)\b|\bv\[(\d+):(\d+)\]')
LABEL = re.compile(r'^(\.LBB\w+|\.Ltmp\w*):')

def regs(text):
    out = set()
    for m in REG.finditer(text):
        if m.group(1): out.add(int(m.group(1)))
        else: out.update(range(int(m.group(2)), int(m.group(3)) + 1))
    return out

def parse(lines):
    """-> list of (kind, text, target) per instruction index, label->index map."""
    ins = []; labels = {}; in_asm = False
    for l in lines:
        s = l.strip()
        if ';;#ASMSTART' in s: in_asm = True; continue
        if ';;#ASMEND' in s: in_asm = False; continue
        m = LABEL.match(s)
        if m: labels[m.group(1)] = len(ins); continue
        t = s.split(';')[0].strip()
        if not t or t.startswith('.') or t.endswith(':'): continue
        ins.append((t, in_asm))
    return ins, labels

def succ(ins, labels, i):
    t = ins[i][0]; op = t.split()[0]
    if op == 's_endpgm': return []
    if op == 's_branch': return [labels[t.split()[1]]]
    if op.startswith('s_cbranch'): return [i + 1, labels[t.split()[1]]]
    if op.startswith('s_setpc') : return []
    return [i + 1]

def check(lines, name):
    ins, labels = parse(lines)
    nload = bad = 0
    for i, (t, asm) in enumerate(ins):
        if not (asm and re.match(r'global_load_dword(x4)?\s', t)): continue
        nload += 1
        d = regs(t.split()[1].rstrip(','))
        seen = set(); q = deque((s, 0) for s in succ(ins, labels, i))
        while q:
            j, cnt = q.popleft()
            if j >= len(ins) or (j, cnt) in seen: continue
            seen.add((j, cnt))
            u = ins[j][0]
            mw = re.match(r's_waitcnt\s+.*vmcnt\((\d+)\)', u)
            if mw and cnt >= int(mw.group(1)): continue          # covered on this path
            ops = u.split(None, 1)
            if len(ops) > 1 and regs(ops[1]) & d:
                print(f"{name}: load #{i} {t.split()[1]} touched before its wait: {u}")
                bad += 1; break
            c2 = min(cnt + (1 if VMEM.match(u) else 0), 64)
            for s in succ(ins, labels, j): q.append((s, c2))
    return nload, bad

def check_file(path, only=None):
    """Returns (loads checked, violations) over the kernels of one assembly file."""
    src = open(path).read().splitlines()
    starts = [i for i, l in enumerate(src) if re.match(r'^_Z\S+:', l)]
    tot = bad = 0
    for k, s0 in enumerate(starts):
        e = starts[k + 1] if k + 1 < len(starts) else len(src)
        name = src[s0].split(':')[0]
        if only and only not in name:
            continue
        n, b = check(src[s0:e], name[-60:])
        tot += n; bad += b
    return tot, bad


if __name__ == "__main__":
    n, b = check_file(sys.argv[1])
    print(f"asm register loads checked: {n}, violations: {b}")
