"""Build-time check of matrix-instruction data hazards in the gfx950 assembly of the kernels.

Some kernels issue v_mfma_f32_32x32x16_bf16 through inline assembly (to choose AGPR or VGPR
operands), so the compiler does not insert the wait states such instructions need.  This
checker walks the final assembly of every kernel and enforces, on all control-flow paths:

R1: the destination registers of an MFMA are not read or written by a non-MFMA instruction,
    nor read as A/B operand by another MFMA, within 12 wait states (a chained accumulation
    into exactly the same registers is allowed back to back);
R2: a register written by a VALU instruction is not read by an MFMA within 2 wait states.

These are the distances the compiler itself keeps for this instruction on gfx950 (its own
output passes the check).  Wait states are counted conservatively: 1 per instruction, 4 per
intervening MFMA, N+1 per s_nop N.  build.py runs the check and fails the build on any violation.
"""
import re, sys

def regs(tok):
    tok = tok.strip()
    m = re.match(r'^([va])\[(\d+):(\d+)\]$', tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r'^([va])(\d+)$', tok)
    if m:
        return {(m.group(1), int(m.group(2)))}
    return set()

def parse(lines):
    ins, labels = [], {}
    for l in lines:
        t = l.split(';')[0].strip()
        if not t:
            continue
        m = re.match(r'^(\.?L\w+|\.LBB\w+):', t)
        if m:
            labels[m.group(1)] = len(ins)
            continue
        if t.startswith('.'):
            continue
        op = t.split()[0]
        rest = t[len(op):].strip()
        args = [a.strip() for a in re.split(r',(?![^\[]*\])', rest)] if rest else []
        ins.append((op, args, t))
    return ins, labels

MEMLOAD = ('ds_read', 'global_load', 'buffer_load', 'scratch_load', 'flat_load', 's_load', 's_buffer_load', 'ds_bpermute')

def dst_src(op, args):
    if op.startswith(('s_', 'global_store', 'buffer_store', 'scratch_store', 'flat_store', 'ds_write')) and not op.startswith('s_nop'):
        srcs = set()
        for a in args:
            srcs |= regs(a)
        return set(), srcs
    if not args:
        return set(), set()
    d = regs(args[0])
    s = set()
    for a in args[1:]:
        s |= regs(a)
    if op.startswith(('global_load_lds', 'buffer_load_lds')):
        return set(), d | s
    return d, s

def ws_of(op, args):
    if op == 's_nop':
        return int(args[0], 0) + 1
    if op.startswith('v_mfma'):
        # an MFMA issues only once the matrix pipe has room: it stands for at least 4 wait
        # states (the pipe takes about 32 cycles per 32x32x16 instruction)
        return 4
    return 1

def succ(ins, labels, i):
    op, args, _ = ins[i]
    out = []
    if op == 's_branch':
        out.append(labels.get(args[0]))
    elif op.startswith('s_cbranch'):
        out.append(labels.get(args[0]))
        out.append(i + 1)
    elif op == 's_endpgm':
        pass
    else:
        out.append(i + 1)
    return [j for j in out if j is not None and j < len(ins)]

def check(lines, name=''):
    ins, labels = parse(lines)
    bad = []
    for i, (op, args, text) in enumerate(ins):
        if op.startswith('v_mfma'):
            D = regs(args[0])
            # walk forward
            stack = [(j, 0) for j in succ(ins, labels, i)]
            seen = set()
            while stack:
                j, ws = stack.pop()
                if ws >= 12 or (j, ws) in seen:
                    continue
                seen.add((j, ws))
                op2, a2, t2 = ins[j]
                d2, s2 = dst_src(op2, a2)
                if op2.startswith('v_mfma'):
                    srcA = regs(a2[1]) if len(a2) > 1 else set()
                    srcB = regs(a2[2]) if len(a2) > 2 else set()
                    srcC = regs(a2[3]) if len(a2) > 3 else set()
                    if (srcA | srcB) & D:
                        bad.append(('R1 mfma->mfma srcAB', ws, text, t2)); continue
                    if srcC & D and not (srcC == D and regs(a2[0]) == D):
                        bad.append(('R1 mfma->mfma srcC partial', ws, text, t2)); continue
                    if d2 & D and not (regs(a2[0]) == D):
                        bad.append(('R1 mfma->mfma WAW', ws, text, t2)); continue
                    if regs(a2[0]) == D:
                        continue   # chained accumulate: the new MFMA is the writer now (checked on its own)
                elif (d2 | s2) & D:
                    bad.append(('R1 mfma->other', ws, text, t2)); continue
                w = ws_of(op2, a2)
                for k in succ(ins, labels, j):
                    stack.append((k, ws + w))
        elif not op.startswith(('v_mfma', 's_')) and not op.startswith(MEMLOAD) and op.startswith('v_'):
            d, _ = dst_src(op, args)
            if not d:
                continue
            stack = [(j, 0) for j in succ(ins, labels, i)]
            seen = set()
            while stack:
                j, ws = stack.pop()
                if ws >= 2 or (j, ws) in seen:
                    continue
                seen.add((j, ws))
                op2, a2, t2 = ins[j]
                if op2.startswith('v_mfma'):
                    s2 = set()
                    for a in a2[1:]:
                        s2 |= regs(a)
                    if s2 & d:
                        bad.append(('R2 valu->mfma', ws, text, t2)); continue
                w = ws_of(op2, a2)
                for k in succ(ins, labels, j):
                    stack.append((k, ws + w))
    return bad

def check_file(path, pattern=''):
    """Returns {kernel symbol: [violations]} for the kernels in an assembly file."""
    s = open(path).read()
    starts = [(m.start(), m.group(1)) for m in re.finditer(r'^(_Z[^:\s]+):', s, re.M)]
    out = {}
    for pos, name in starts:
        if pattern not in name:
            continue
        end = s.find('.Lfunc_end', pos)
        out[name] = check(s[pos:end].split('\n'), name)
    return out


if __name__ == '__main__':
    res = check_file(sys.argv[1], sys.argv[2] if len(sys.argv) > 2 else '')
    total = 0
    for name, bad in res.items():
        total += len(bad)
        print(f'{name[:90]}: {len(bad)} violations')
        for b in bad[:8]:
            print('   ', b)
    sys.exit(1 if total else 0)
