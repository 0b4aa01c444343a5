"""Path-aware check of the wait states between an MFMA and the first
instruction that reads its result, over the gfx950 assembly of the library's
own sources.

The compiler's hazard recognizer inserts the wait states (instructions issued
in between plus ``s_nop`` counts) that an MFMA's result needs before a VALU or
memory instruction may read it.  On a straight-line path it always does; where
a conditional branch sits between the MFMA and the read, it has been seen to
count the instructions of the skipped block, leaving the other path short, and
the read then sees a partial accumulator.  This module walks every path from
each MFMA to the first reader of its destination and reports any path with
fewer wait states than the compiler itself places, for the same opcode and the
same kind of reader, where all paths agree.
"""
from __future__ import annotations

import os
import re
import subprocess

_RANGE = re.compile(r"([va])\[(\d+):(\d+)\]$")
_SINGLE = re.compile(r"([va])(\d+)$")
_STORES = ("global_store", "buffer_store", "ds_write", "ds_store", "flat_store", "scratch_store")


def _regs(tok: str) -> set:
    tok = tok.strip()
    m = _RANGE.match(tok)
    if m:
        return {(m.group(1), k) for k in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = _SINGLE.match(tok)
    if m:
        return {(m.group(1), int(m.group(2)))}
    return set()


def _split(ins: str):
    p = ins.split(None, 1)
    if len(p) < 2:
        return p[0], []
    return p[0], [o.strip() for o in p[1].split(",")]


def _reads(ins: str) -> set:
    op, o = _split(ins)
    src = o if op.startswith(_STORES) else o[1:]
    out = set()
    for x in src:
        out |= _regs(x)
    return out


def parse(asm: str):
    """Instructions, label -> index, and (index, function name) starts."""
    ins, labels, funcs = [], {}, []
    for ln in asm.split("\n"):
        s = ln.split(";")[0].strip()
        if not s:
            continue
        if s.endswith(":"):
            if s.startswith(".L"):
                labels[s[:-1]] = len(ins)
            elif not s.startswith("."):
                funcs.append((len(ins), s[:-1]))
            continue
        if s.startswith("."):
            continue
        ins.append(s)
    return ins, labels, funcs


def mfma_read_waits(asm: str, horizon: int = 64):
    """For each MFMA and each path to a reader of its destination: (function,
    instruction, opcode, reader kind, wait states, branch crossed, whether an
    ``s_nop`` directly precedes the reader)."""
    ins, labels, funcs = parse(asm)
    out = []
    for i, t in enumerate(ins):
        if not t.startswith("v_mfma"):
            continue
        op, o = _split(t)
        dst = _regs(o[0])
        fn = [f for s, f in funcs if s <= i][-1] if funcs else "?"
        seen = set()
        stack = [(i + 1, 0, False)]
        while stack:
            pc, w, br = stack.pop()
            while pc < len(ins) and w <= horizon:
                u = ins[pc]
                kind = None
                if u.startswith("v_mfma"):
                    uo = _split(u)[1]
                    if len(uo) > 3 and _regs(uo[3]) & dst:
                        break                       # accumulation chain: interlocked
                    if (_regs(uo[1]) | _regs(uo[2])) & dst:
                        kind = "mfma"
                elif _reads(u) & dst:
                    kind = "other"
                if kind:
                    nop = pc > 0 and ins[pc - 1].startswith("s_nop")
                    out.append((fn, t, op, kind, w, br, nop))
                    break
                w += int(u.split()[1]) + 1 if u.startswith("s_nop") else 1
                if u.startswith("s_endpgm"):
                    break
                if u.startswith("s_branch"):
                    pc, br = labels[u.split()[1]], True
                    continue
                if u.startswith("s_cbranch"):
                    br = True
                    tgt = labels.get(u.split()[1])
                    if tgt is not None and (tgt, w) not in seen:
                        seen.add((tgt, w))
                        stack.append((tgt, w, True))
                pc += 1
    return out


def short_paths(asm: str):
    """Paths through a branch that reach a reader of an MFMA result with fewer
    wait states than the compiler pads a straight path to (an ``s_nop``
    directly before the reader) for the same opcode and reader kind, or, for
    an opcode never padded, than its shortest straight path."""
    rows = mfma_read_waits(asm)
    padded, straight = {}, {}
    for fn, t, op, kind, w, br, nop in rows:
        if not br:
            straight[(op, kind)] = min(straight.get((op, kind), 1 << 30), w)
            if nop:
                padded[(op, kind)] = min(padded.get((op, kind), 1 << 30), w)
    need = {**straight, **padded}
    bad = []
    for fn, t, op, kind, w, br, nop in rows:
        n = need.get((op, kind))
        if br and n is not None and w < n:
            bad.append((fn, t, kind, w, n))
    return bad, need


def device_asm(src: str, hipcc: str, flags: list) -> str:
    """gfx950 device assembly of one source file, built with the library's flags."""
    keep = [f for f in flags if f not in ("-shared", "-fPIC")]
    r = subprocess.run([hipcc] + keep + ["--cuda-device-only", "-S", "-o", "-", "-x", "hip", src],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc -S {os.path.basename(src)} failed:\n{r.stderr[-2000:]}")
    return r.stdout
