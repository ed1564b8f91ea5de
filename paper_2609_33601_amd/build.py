"""Build libjq.so (the gfx950 HIP library behind include/jq.h) in-tree with hipcc.

Each source compiles to its own object in parallel (_build/), then one hipcc
link makes the shared library.  Every call compiles every source.  Alongside,
the BF6 kernels are compiled to device assembly once more and the GEMM's
hand-ordered vector loads are checked against their waits (check_waits.py); a
failed check fails the build.
"""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

try:
    from . import check_waits
except ImportError:  # run as a script
    import check_waits

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJ_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libjq.so")
SOURCES = ["quantize.hip", "ternary.hip", "gemm.hip", "gemm_group.hip", "f6.hip", "jq_api.cpp"]
ARCH = "gfx950"

# Per-source flags: the BF6 kernels are built without machine sinking, which
# would move the first k-step's MFMAs of a GEMM stage below its barrier.
SOURCE_FLAGS = {"f6.hip": ["-mllvm", "-disable-machine-sink"]}
# Sources whose asm-issued loads are checked against their waits, and the
# kernel names checked in each.
CHECKED_SOURCES = {"f6.hip": "w4a4_f6_gemm_kernel"}

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # every fp32 operation of the quantiser and the epilogue is rounded on its own
    "-ffp-contract=off",
    # no packed-fp32 VALU instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def build(verbose=False, extra_flags=(), jobs=None):
    """Compile the library; returns the path of the built .so."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    cc = hipcc()
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    objs = [os.path.join(OBJ_DIR, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    cmds = [[cc, *HIPCC_FLAGS, *SOURCE_FLAGS.get(s, []), *extra_flags, *inc, "-c", os.path.join(CSRC, s), "-o", o]
            for s, o in zip(SOURCES, objs)]
    checked = [s for s in SOURCES if s in CHECKED_SOURCES]
    jobs = jobs or max(1, min(len(cmds) + len(checked), os.cpu_count() or 1))
    with ThreadPoolExecutor(max_workers=jobs) as pool:
        futs = [pool.submit(_run, c, verbose) for c in cmds]
        futs += [pool.submit(check_waits.compile_and_check,
                             [cc, *HIPCC_FLAGS, *SOURCE_FLAGS.get(s, []), *extra_flags, *inc],
                             os.path.join(CSRC, s), os.path.join(OBJ_DIR, os.path.splitext(s)[0] + ".s"),
                             CHECKED_SOURCES[s])
                 for s in checked]
        for f in futs:
            f.result()
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
