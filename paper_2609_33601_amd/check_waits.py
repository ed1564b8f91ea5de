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

The scan is linear over each kernel's text and runs twice round it (the stage
loop's back edge).  Loads into LDS (``... lds``) have no destination
registers; stores and scratch accesses count towards vmcnt like loads.
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


def hazards(lines):
    """Instructions of one kernel that touch a possibly pending load's destination.

    Returns (line number, instruction, line number of the load) triples."""
    pending = []  # vector-memory operations in issue order: (line, destination registers)
    found = {}
    for _ in range(2):
        for ln, text in lines:
            s = text.split(";")[0].strip()
            if not s or s.endswith(":") or s.startswith("."):
                continue
            op = s.split()[0]
            args = s[len(op):]
            if op == "s_waitcnt":
                m = _VMCNT.search(args)
                if m:
                    n = int(m.group(1))
                    pending = pending[len(pending) - n:] if n else []
                continue
            is_vmem = op.startswith(_VMEM_PREFIXES)
            parts = [a.strip() for a in args.split(",")]
            is_load = is_vmem and "load" in op and not re.search(r"\blds\b", args)
            dest = registers(parts[0]) if is_load else set()
            used = set()
            for p in (parts[1:] if is_load else parts):
                used |= registers(p)
            for load_ln, load_dest in pending:
                if load_dest & used:
                    found[(ln, load_ln)] = s
            if is_vmem:
                pending.append((ln, dest))
    return [(ln, s, load_ln) for (ln, load_ln), s in sorted(found.items())]


def kernels(asm_text, pattern):
    """(name, [(line number, text)]) of every kernel whose symbol matches `pattern`."""
    src = asm_text.split("\n")
    out = []
    i = 0
    while i < len(src):
        m = re.match(r"^(_Z\S*" + pattern + r"\S*):", src[i])
        if m:
            j = i
            while j < len(src) and "s_endpgm" not in src[j]:
                j += 1
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


def compile_and_check(cmd_prefix, source, out_asm):
    """Compile `source` to device assembly with the given hipcc command prefix and check it."""
    res = subprocess.run([*cmd_prefix, "--cuda-device-only", "-S", source, "-o", out_asm],
                         stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc -S failed ({res.returncode}) for {source}\n{res.stdout}")
    with open(out_asm) as f:
        return check_asm(f.read())


if __name__ == "__main__":
    with open(sys.argv[1]) as f:
        print(f"{check_asm(f.read())} kernels checked")
