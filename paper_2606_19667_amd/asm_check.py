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
of its own; `s_waitcnt vmcnt(k)` covers a load on a path where at least k
memory instructions were issued after it.
"""
from __future__ import annotations

import re

_VMEM = re.compile(r'^(global_|buffer_|flat_|scratch_)')
_LOAD = re.compile(r'^global_load_dword(x[234])?\s')
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


def parse(lines: list[str]):
    """Instructions (text), label -> instruction index, and the indices of
    untracked loads."""
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
                    untracked.extend(i for i in block if _LOAD.match(insts[i]))
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


def _successors(insts, labels, i):
    op = insts[i].split()[0]
    if op == 's_endpgm':
        return []
    if op == 's_branch':
        return [labels[insts[i].split()[1]]]
    if op.startswith('s_cbranch'):
        return [labels[insts[i].split()[1]], i + 1]
    return [i + 1]


def hazards(lines: list[str]) -> list[tuple[str, str]]:
    """(load, offending instruction) pairs over every path of one function."""
    insts, labels, loads = parse(lines)
    found = []
    for li in loads:
        dst = vregs(insts[li].split()[1].rstrip(','))
        seen = set()
        stack = [(li + 1, 0)]
        while stack:
            i, younger = stack.pop()
            if i >= len(insts):
                continue
            key = (i, min(younger, 64))
            if key in seen:
                continue
            seen.add(key)
            text = insts[i]
            op = text.split()[0]
            if op == 's_waitcnt':
                m = re.search(r'vmcnt\((\d+)\)', text)
                if m and int(m.group(1)) <= younger:
                    continue
            elif op == 's_barrier':
                continue
            elif vregs(text) & dst:
                found.append((insts[li], text))
                continue
            nxt = younger + (1 if _VMEM.match(text) else 0)
            for s in _successors(insts, labels, i):
                stack.append((s, nxt))
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
