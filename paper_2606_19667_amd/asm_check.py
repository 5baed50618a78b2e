"""Build-time check of the attention kernels' assembly for untracked loads.

The attention kernel issues some global loads through inline asm so that the
compiler does not track them (a tracked load makes it wait for every
load-to-LDS copy in flight before the first use). Their results are complete
only after a later `s_waitcnt vmcnt(n)` that covers them, or a step barrier
(whose wait leaves only the copies issued after them in flight). Until then the
destination registers must not be read or written: the compiler does not know
that, so this check walks every control-flow path of the generated gfx9
assembly from each such load and reports any instruction that touches its
destination registers before a covering wait.

A load counts as untracked when it sits in an inline-asm block without a wait
of its own; `s_waitcnt vmcnt(k)` covers a vector load on a path where at least
k memory instructions were issued after it. Untracked scalar loads
(`s_load_dword*`, SGPR destinations) are covered only by an `s_waitcnt` with
`lgkmcnt(0)` (scalar loads return out of order).

Paths follow branch conditions in one form the compiler uses for wave-uniform
if/else: an if/else becomes two sequential `if`s on one SGPR-pair flag F set
to all lanes (-1) or none (0) by s_mov_b64, each testing `vcc = exec & F` (or
`exec & ~F`) with s_cbranch_vccz/vccnz. A path knows F from its last constant
assignment until an instruction writes F, and takes only the branch direction
that value gives (exec is taken to be nonzero). Flags of any other origin (a
per-lane compare, say) are not evaluated: both directions are followed.
"""
from __future__ import annotations

import re

_VMEM = re.compile(r'^(global_|buffer_|flat_|scratch_)')
_LOAD = re.compile(r'^global_load_dword(x[234])?\s')
_SLOAD = re.compile(r'^s_load_dword(x[248])?\s')
_SREG = re.compile(r'\bs\[(\d+):(\d+)\]|\bs(\d+)\b')
_LABEL = re.compile(r'^(\.?[\w.$]+):')
_VREG = re.compile(r'\bv\[(\d+):(\d+)\]|\bv(\d+)\b')


def vregs(text: str) -> set[int]:
    """VGPR numbers named in an instruction's text."""
    out: set[int] = set()
    for m in _VREG.finditer(text):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def sregs(text: str) -> set[int]:
    """SGPR numbers named in an instruction's operands."""
    out: set[int] = set()
    parts = text.split(None, 1)
    if len(parts) < 2:
        return out
    for m in _SREG.finditer(parts[1]):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def parse(lines: list[str]):
    """Instructions (text), label -> instruction index, and the indices of
    untracked loads (vector and scalar)."""
    insts: list[str] = []
    labels: dict[str, int] = {}
    untracked: list[int] = []
    block: list[int] | None = None
    for raw in lines:
        if ';;#ASMSTART' in raw:
            block = []
            continue
        if ';;#ASMEND' in raw:
            if block is not None:
                texts = [insts[i] for i in block]
                if not any(t.startswith('s_waitcnt') for t in texts):
                    untracked.extend(i for i in block if _LOAD.match(insts[i]) or _SLOAD.match(insts[i]))
            block = None
            continue
        text = raw.split(';')[0].strip()
        if not text:
            continue
        m = _LABEL.match(text)
        if m:
            labels[m.group(1)] = len(insts)
            continue
        if text.startswith('.'):
            continue
        if block is not None:
            block.append(len(insts))
        insts.append(text)
    return insts, labels, untracked


_SPAIR = re.compile(r'^s\[(\d+):(\d+)\]$')
_SREG1 = re.compile(r'^s(\d+)$')
# mnemonics whose first operand is not a register they write
_NO_DEST = ('s_cmp', 's_bitcmp', 's_cbranch', 's_branch', 's_waitcnt', 's_barrier', 's_nop', 's_endpgm',
            's_setprio', 's_sleep', 's_sendmsg', 'global_store', 'buffer_store', 'ds_write', 'scratch_store')


def _operands(text: str) -> list[str]:
    parts = text.split(None, 1)
    return [x.strip() for x in parts[1].split(',')] if len(parts) > 1 else []


def _sdest(text: str) -> set[int] | None:
    """SGPR numbers an instruction writes through its first operand; None when
    it writes vcc (as a first operand or implicitly, v_cmp*_e32)."""
    op = text.split()[0]
    if op.startswith('v_cmp') and op.endswith('_e32'):
        return None
    if op.startswith(_NO_DEST):
        return set()
    ops = _operands(text)
    if not ops:
        return set()
    first = ops[0]
    if first == 'vcc':
        return None
    m = _SPAIR.match(first)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = _SREG1.match(first)
    if m:
        return {int(m.group(1))}
    return set()


def _vcc_flag(text: str):
    """(F, negated) when the instruction is `s_and_b64 vcc, exec, F` or
    `s_andn2_b64 vcc, exec, F` with F an SGPR pair, else None."""
    op = text.split()[0]
    if op not in ('s_and_b64', 's_andn2_b64'):
        return None
    ops = _operands(text)
    if len(ops) != 3 or ops[0] != 'vcc' or ops[1] != 'exec':
        return None
    m = _SPAIR.match(ops[2])
    if not m:
        return None
    return (int(m.group(1)), int(m.group(2))), op == 's_andn2_b64'


def _successors(insts, labels, i):
    op = insts[i].split()[0]
    if op == 's_endpgm':
        return []
    if op == 's_branch':
        return [labels[insts[i].split()[1]]]
    if op.startswith('s_cbranch'):
        return [labels[insts[i].split()[1]], i + 1]
    return [i + 1]


def _step(insts, labels, i, vflag, known):
    """Successor states (instruction, vflag, known) of instruction i: the flag
    tests of s_cbranch_vccz/vccnz, and forgetting flags an instruction writes."""
    text = insts[i]
    op = text.split()[0]
    if op in ('s_cbranch_vccz', 's_cbranch_vccnz') and vflag is not None:
        flag, neg = vflag
        taken_f = (not neg) if op == 's_cbranch_vccnz' else neg   # F under which the branch is taken
        kv = dict(known)
        out = []
        for succ, fval in ((labels[text.split()[1]], taken_f), (i + 1, not taken_f)):
            if flag in kv and kv[flag] != fval:
                continue
            out.append((succ, vflag, known))
        return out
    f = _vcc_flag(text)
    if f is not None:
        vflag = f
    else:
        w = _sdest(text)
        if w is None:
            vflag = None
        elif w:
            known = frozenset(x for x in known if not (set(range(x[0][0], x[0][1] + 1)) & w))
            if vflag is not None and set(range(vflag[0][0], vflag[0][1] + 1)) & w:
                vflag = None
            # a flag set to a constant: all lanes (-1) or none (0)
            ops = _operands(text)
            m = _SPAIR.match(ops[0]) if op == 's_mov_b64' and len(ops) == 2 else None
            if m and ops[1] in ('-1', '0'):
                known = known | {((int(m.group(1)), int(m.group(2))), ops[1] == '-1')}
    return [(s, vflag, known) for s in _successors(insts, labels, i)]


def _entry_facts(insts, labels):
    """For each instruction, the (vflag, known flags) that hold on every path
    from the function's entry to it (None: unreachable)."""
    state: list = [None] * len(insts)
    if not insts:
        return state
    state[0] = (None, frozenset())
    work = [0]
    while work:
        i = work.pop()
        if i >= len(insts) or state[i] is None:
            continue
        vflag, known = state[i]
        for succ, v2, k2 in _step(insts, labels, i, vflag, known):
            if succ >= len(insts):
                continue
            old = state[succ]
            new = (v2, k2) if old is None else (old[0] if old[0] == v2 else None, old[1] & k2)
            if new != old:
                state[succ] = new
                work.append(succ)
    return state


def hazards(lines: list[str]) -> list[tuple[str, str]]:
    """(load, offending instruction) pairs over every feasible path of one
    function (feasible as far as the flag tests described above tell)."""
    insts, labels, loads = parse(lines)
    facts = _entry_facts(insts, labels)
    found = []
    for li in loads:
        scalar = bool(_SLOAD.match(insts[li]))
        first = insts[li].split()[1].rstrip(',')
        dst = sregs('x ' + first) if scalar else vregs(first)
        touches = sregs if scalar else vregs
        if facts[li] is None:
            continue
        seen = set()
        # (instruction, memory instructions issued since the load, the flag the
        # last vcc write tests, known flag values)
        stack = [(s, 0, v, k) for s, v, k in _step(insts, labels, li, *facts[li])]
        while stack:
            i, younger, vflag, known = stack.pop()
            if i >= len(insts):
                continue
            key = (i, min(younger, 64), vflag, known)
            if key in seen:
                continue
            seen.add(key)
            text = insts[i]
            op = text.split()[0]
            if op == 's_waitcnt':
                if scalar:
                    if re.search(r'lgkmcnt\(0\)', text):
                        continue
                else:
                    m = re.search(r'vmcnt\((\d+)\)', text)
                    if m and int(m.group(1)) <= younger:
                        continue
            elif op == 's_barrier' and not scalar:
                continue
            elif touches(text) & dst:
                found.append((insts[li], text))
                continue
            nxt = younger + (1 if _VMEM.match(text) else 0)
            for s, v2, k2 in _step(insts, labels, i, vflag, known):
                stack.append((s, nxt, v2, k2))
    return found


def functions(asm_text: str, name_part: str) -> dict[str, list[str]]:
    """Lines of every function whose symbol contains name_part."""
    lines = asm_text.split('\n')
    out = {}
    for i, line in enumerate(lines):
        m = re.match(r'^([A-Za-z_][\w.$]*):', line)
        if m and name_part in m.group(1) and not m.group(1).startswith('.'):
            end = next((j for j in range(i, len(lines)) if lines[j].startswith('.Lfunc_end')), len(lines))
            out[m.group(1)] = lines[i:end + 1]
    return out


def check(asm_text: str, name_part: str = 'suffix_prefill_attn_kernel') -> dict[str, int]:
    """Untracked loads per checked function; raises on any hazard."""
    report = {}
    for name, lines in functions(asm_text, name_part).items():
        bad = hazards(lines)
        if bad:
            raise RuntimeError(f"{name}: destination of an untracked load used before its wait: {bad[:4]}")
        report[name] = len(parse(lines)[2])
    if not report:
        raise RuntimeError(f"no function matching {name_part!r} in the assembly")
    return report
