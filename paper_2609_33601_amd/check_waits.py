"""Build-time check of the BF6 GEMM's hand-ordered vector loads.

The BF6 GEMM issues its weight loads as inline asm and orders them with
explicit s_waitcnt instructions.  The compiler does not know that an asm
load completes later than it is issued, so nothing but the kernel's own
structure keeps it from reading, copying or spilling a load's destination
registers before the wait that retires the load.  This module reads the AMD
assembly of the kernels built here and fails the build if any instruction
touches the destination registers of a vector-memory load that, by the
in-order completion of vector loads and the vmcnt waits in between, may still
be in flight.

The check follows the kernel's control flow: its text is cut into basic
blocks at labels and branches, and the vector-memory operations that may be
in flight are carried along every edge to a fixed point, each with the least
number of younger operations issued after it on any path (a vmcnt(N) wait
retires a load once at least N younger operations follow it).  Loads into
LDS (``... lds``) have no destination registers; stores and scratch accesses
count towards vmcnt like loads.
"""

import re
import subprocess
import sys

_RANGE = re.compile(r"\b([va])\[(\d+):(\d+)\]")
_SINGLE = re.compile(r"\b([va])(\d+)\b")
_VMCNT = re.compile(r"vmcnt\((\d+)\)")
_VMEM_PREFIXES = ("buffer_", "global_", "scratch_")


def registers(text):
    """The vector registers (('v'|'a', index)) named in an operand string."""
    out = set()
    for m in _RANGE.finditer(text):
        out |= {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    for m in _SINGLE.finditer(_RANGE.sub("", text)):
        out.add((m.group(1), int(m.group(2))))
    return out


_LABEL = re.compile(r"^(\.?L\w+|_Z\S+):")
_BB_COMMENT = re.compile(r"^;\s*%bb\.\d+:")
_YOUNGER_CAP = 64  # above any vmcnt immediate


def _blocks(lines):
    """Basic blocks of one kernel: a list of [labels, instructions, successors].

    Successors are block indices; instructions are (line number, text)."""
    blocks, label_at = [], {}
    cur = [[], [], None]  # labels, instructions, successor spec

    def close(spec):
        nonlocal cur
        cur[2] = spec
        blocks.append(cur)
        cur = [[], [], None]

    for ln, text in lines:
        raw = text.split(";")[0].strip() if not _BB_COMMENT.match(text.strip()) else ""
        m = _LABEL.match(text.strip())
        if m or _BB_COMMENT.match(text.strip()):
            if cur[1]:
                close(("fall",))
            if m:
                cur[0].append(m.group(1))
            continue
        if not raw or raw.startswith("."):
            continue
        op = raw.split()[0]
        cur[1].append((ln, raw))
        if op == "s_branch":
            close(("to", raw.split()[1]))
        elif op.startswith("s_cbranch"):
            close(("to", raw.split()[1], "fall"))
        elif op in ("s_endpgm", "s_setpc_b64") or op.startswith("s_endpgm"):
            close(("end",))
    if cur[1] or cur[0]:
        close(("end",))
    for i, b in enumerate(blocks):
        for name in b[0]:
            label_at[name] = i
    for i, b in enumerate(blocks):
        spec, succ = b[2], []
        if spec[0] == "fall":
            succ = [i + 1] if i + 1 < len(blocks) else []
        elif spec[0] == "to":
            if spec[1] in label_at:
                succ.append(label_at[spec[1]])
            if len(spec) > 2 and i + 1 < len(blocks):
                succ.append(i + 1)
        b[2] = succ
    return blocks


def _step(state, ln, s, found):
    """Apply one instruction to the in-flight state {load line: (dest, younger)}."""
    op = s.split()[0]
    args = s[len(op):]
    if op == "s_waitcnt":
        m = _VMCNT.search(args)
        if m:
            n = int(m.group(1))
            state = {k: v for k, v in state.items() if v[1] < n}
        return state
    is_vmem = op.startswith(_VMEM_PREFIXES)
    parts = [a.strip() for a in args.split(",")]
    is_load = is_vmem and "load" in op and "lds" not in op and not re.search(r"\blds\b", args)
    dest = registers(parts[0]) if is_load else set()
    used = set()
    for p in (parts[1:] if is_load else parts):
        used |= registers(p)
    for load_ln, (load_dest, _) in state.items():
        if load_dest & used:
            found[(ln, load_ln)] = s
    if is_vmem:
        state = {k: (d, min(y + 1, _YOUNGER_CAP)) for k, (d, y) in state.items()}
        if dest:
            state[ln] = (frozenset(dest), 0)
    return state


def _merge(a, b):
    out = dict(a)
    for k, (d, y) in b.items():
        out[k] = (d, min(y, out[k][1])) if k in out else (d, y)
    return out


def hazards(lines):
    """Instructions of one kernel that touch a possibly pending load's destination.

    Returns (line number, instruction, line number of the load) triples."""
    blocks = _blocks(lines)
    if not blocks:
        return []
    entry = [None] * len(blocks)
    entry[0] = {}
    found = {}
    work = [0]
    while work:
        i = work.pop()
        state = entry[i]
        for ln, s in blocks[i][1]:
            state = _step(state, ln, s, found)
        for j in blocks[i][2]:
            new = state if entry[j] is None else _merge(entry[j], state)
            if new != entry[j]:
                entry[j] = new
                work.append(j)
    return [(ln, s, load_ln) for (ln, load_ln), s in sorted(found.items())]


def kernels(asm_text, pattern):
    """(name, [(line number, text)]) of every kernel whose symbol matches `pattern`.

    A kernel's text runs from its symbol to its .Lfunc_end label (blocks may
    follow an s_endpgm), or to the last s_endpgm before the next symbol."""
    src = asm_text.split("\n")
    out = []
    i = 0
    while i < len(src):
        m = re.match(r"^(_Z\S*" + pattern + r"\S*):", src[i])
        if m:
            j, last_end = i + 1, None
            while j < len(src) and not re.match(r"^\.Lfunc_end\d+:", src[j]) and not re.match(r"^_Z\S*:", src[j]):
                if "s_endpgm" in src[j]:
                    last_end = j
                j += 1
            if j >= len(src) or not src[j].startswith(".Lfunc_end"):
                j = last_end if last_end is not None else j - 1
            out.append((m.group(1), list(enumerate(src[i:j + 1], start=i + 1))))
            i = j
        i += 1
    return out


def check_asm(asm_text, pattern="w4a4_f6_gemm_kernel"):
    """Raise RuntimeError naming the first hazards found in the matching kernels."""
    ks = kernels(asm_text, pattern)
    if not ks:
        raise RuntimeError(f"no kernel matching {pattern!r} in the assembly")
    problems = []
    for name, lines in ks:
        for ln, ins, load_ln in hazards(lines):
            problems.append(f"{name}: line {ln} '{ins}' touches the registers of the load at line {load_ln}")
    if problems:
        raise RuntimeError("vector-load ordering check failed:\n" + "\n".join(problems[:10]))
    return len(ks)


def compile_and_check(cmd_prefix, source, out_asm, pattern="w4a4_f6_gemm_kernel"):
    """Compile `source` to device assembly with the given hipcc command prefix and check
    the kernels whose names match `pattern`."""
    res = subprocess.run([*cmd_prefix, "--cuda-device-only", "-S", source, "-o", out_asm],
                         stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc -S failed ({res.returncode}) for {source}\n{res.stdout}")
    with open(out_asm) as f:
        return check_asm(f.read(), pattern)


if __name__ == "__main__":
    with open(sys.argv[1]) as f:
        print(f"{check_asm(f.read(), *sys.argv[2:3])} kernels checked")
