"""Build-time check of LDS reads issued from inline assembly.

Some kernels issue ds_read instructions from inline assembly and wait for
them (s_waitcnt lgkmcnt) in a later asm statement, so that the reads of the
next block overlap the matrix-core work of the current one.  Between the read
and the wait the compiler believes the destination registers already hold
their final value; if it copied, spilled or reused one of them there, the
kernel would read stale data.  This module checks the AMD GCN assembly that
the compiler actually produced: for every ds_read* of every kernel, on every
control-flow path from the read, no instruction may name any of the read's
destination registers before an s_waitcnt lgkmcnt(k) with k at most the number
of LDS instructions issued after the read on that path (LDS instructions
complete in order, so the read has then completed).  A later LDS read may
write registers of an earlier one (its data lands last); its address may not
name them.  Every branch is followed both ways, so the check is conservative.

build.py runs it on the device assembly of the sources whose kernels use such
split reads; a kernel that fails is compiled out of use (its launcher falls
back to a kernel whose reads the compiler tracks or that waits inside the
same asm statement).  `python -m paper_1802_00930_amd.asm_check FILE.s`
prints the report.
"""
from __future__ import annotations

import re
import subprocess
import sys
from typing import Dict, List, Set, Tuple

_REG = re.compile(r"\b([va])(?:\[(\d+):(\d+)\]|(\d+)\b)")
_LABEL = re.compile(r"^([.\w$]+):")
_LGKM = re.compile(r"lgkmcnt\((\d+)\)")


def _regs(operands: str) -> Set[Tuple[str, int]]:
    out = set()
    for m in _REG.finditer(operands):
        kind = m.group(1)
        if m.group(4) is not None:
            out.add((kind, int(m.group(4))))
        else:
            for r in range(int(m.group(2)), int(m.group(3)) + 1):
                out.add((kind, r))
    return out


def _functions(text: str) -> Dict[str, List[str]]:
    """Kernel name -> its instruction / label lines (comments stripped)."""
    funcs, cur, body = {}, None, []
    for raw in text.splitlines():
        line = raw.split(";")[0].rstrip()
        if not line.strip():
            continue
        m = _LABEL.match(line)
        if m and not line.startswith(".") and not line.startswith("\t"):
            name = m.group(1)
            if name.startswith("_Z") or name.startswith("__"):
                if cur:
                    funcs[cur] = body
                cur, body = name, []
                continue
        if cur is None:
            continue
        s = line.strip()
        if s.startswith(".Lfunc_end") or s == "s_endpgm":
            body.append("s_endpgm")
            if s.startswith(".Lfunc_end"):
                funcs[cur] = body
                cur, body = None, []
            continue
        if s.startswith(".") and not _LABEL.match(s):
            continue  # directives
        body.append(s)
    if cur:
        funcs[cur] = body
    return funcs


def _cfg(body: List[str]):
    labels = {}
    for i, s in enumerate(body):
        m = _LABEL.match(s)
        if m:
            labels[m.group(1)] = i
    return labels


def _successors(body, labels, i):
    s = body[i]
    op = s.split()[0]
    if op == "s_endpgm":
        return []
    if op.startswith("s_branch"):
        return [labels[s.split()[1]]]
    if op.startswith("s_cbranch"):
        return [labels[s.split()[1]], i + 1]
    if op in ("s_setpc_b64", "s_swappc_b64"):
        return None  # indirect: not analysable
    return [i + 1] if i + 1 < len(body) else []


def check_function(body: List[str]) -> List[str]:
    """Violations: read line, offending line."""
    labels = _cfg(body)
    problems = []
    for i, s in enumerate(body):
        op = s.split()[0]
        if not op.startswith("ds_read"):
            continue
        dest0 = frozenset(_regs(s[len(op):].split(",")[0]))
        if not dest0:
            continue
        seen = set()
        stack = [(i + 1, 0, dest0)]
        while stack:
            state = stack.pop()
            j, n_after, dest = state
            if j >= len(body) or not dest or state in seen:
                continue
            seen.add(state)
            t = body[j]
            if _LABEL.match(t):
                stack.append((j + 1, n_after, dest))
                continue
            top = t.split()[0]
            if top == "s_waitcnt":
                m = _LGKM.search(t)
                if m and int(m.group(1)) <= n_after:
                    continue  # the read has completed on this path
            parts = t[len(top):].split(",")
            if top.startswith("ds_read"):
                # a later LDS read may reuse registers of this one (LDS reads
                # return in order, so its data lands last); its address must not
                if _regs(",".join(parts[1:])) & dest:
                    problems.append("%s  ->  %s" % (s, t))
                    continue
                dest = dest - frozenset(_regs(parts[0]))
            elif _regs(t[len(top):]) & dest:
                problems.append("%s  ->  %s" % (s, t))
                continue
            n2 = min(n_after + (1 if top.startswith("ds_") else 0), 64)
            succ = _successors(body, labels, j)
            if succ is None:
                problems.append("%s  ->  indirect branch %s" % (s, t))
                continue
            for k in succ:
                stack.append((k, n2, dest))
    return problems


def check_text(text: str) -> Dict[str, List[str]]:
    return {name: check_function(body) for name, body in _functions(text).items()}


def demangle(names):
    try:
        res = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True,
                             text=True, check=True)
        return dict(zip(names, res.stdout.splitlines()))
    except (OSError, subprocess.CalledProcessError):
        return {n: n for n in names}


if __name__ == "__main__":
    rep = check_text(open(sys.argv[1]).read())
    dm = demangle(list(rep))
    bad = 0
    for name, probs in sorted(rep.items()):
        print("%-6s %s" % ("FAIL" if probs else "ok", dm[name]))
        for p in probs[:5]:
            print("        " + p)
        bad += bool(probs)
    sys.exit(1 if bad else 0)
